// Distribute + PointNet + per-vertex max, fused (Sec. "Proposed Operations":
// Distribute, Eq. distribute; the PointNet block of the network figure;
// Sec. "Performance" suggests fusing Distribute and the PointNet into one
// operation so that the distributed rows are never stored).
//
// Every pair (point p, simplex vertex v) of the last splat is one row:
//   h_0 = [g_p - mu_v ; f_p]          (D_G: position minus the local mean
//                                      mu_v of J_v; D_F: the features)
//   h_l = W_l relu(N_l(h_{l-1})) + b_l,   l = 1, 2, 3, widths 16, 32, 64
//   x_v = max over the rows of v of h_3, per channel.
// N_l is a group normalisation (Sec. "Implementation": every convolution is
// pre-activated by group normalisation and ReLU): per cloud (batch id) and
// group of channels, the mean and variance over all the cloud's rows, then
// per channel gamma (h - mean) / sqrt(var + eps) + beta.  Once the statistics
// are known N_l is a per-channel affine a h + s, which is how the kernels
// apply it; a caller may also give (a, s) directly (no statistics).
//
// The rows are the entries of the splat's pair lists, which are grouped by
// vertex, so the rows of one vertex are consecutive:
//   k_entry_vertex   entry -> vertex map (one thread per short list, one per
//                    32-entry part of a long list, as the splat's gather);
//                    also zeroes the vertex's fp64 position sum, and finds
//                    the number of batch ids (clouds) of a batched lattice
//   k_local_mean     one lane per entry; each wavefront owns 64 consecutive
//                    entries and sums the positions of each run of equal
//                    vertex in fp64 (a segmented scan over shuffles); a run
//                    that is the vertex's whole list writes mu_v, otherwise
//                    the run is added to the vertex's fp64 sum atomically
//   k_pointnet_prep  mu_v of the lists that cross a 64-entry chunk; the key
//                    of -inf in the key row of each vertex whose list crosses
//                    a chunk boundary; the parameters in the padded layout;
//                    the statistics rows zeroed (independent jobs in one
//                    launch)
//   with group normalisation, three statistics passes, each followed by
//   k_gn_finalize, which turns the sums of the block's input into the
//   affine (a, s) per cloud and channel:
//     k_gn_stats0    h_0 per entry: per cloud, the row count and the fp64
//                    sums of h_0 and h_0^2 per channel
//     k_pointnet<1>  block 1 per entry: the sums of h_1 and h_1^2
//     k_pointnet<2>  blocks 1 and 2: the sums of h_2 and h_2^2
//   k_pointnet<3>    the three blocks as fp32 MFMA products over the
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
//   k_pointnet_rows  the crossing lists' keys decoded into their rows.
// The statistics are fp64 sums added with atomics (their order varies from
// run to run by a few fp64 ulps, far below the fp32 results' rounding).
#include "internal.h"
#include "rowsum.h"

namespace {

constexpr int kBlock = 256;
constexpr int kWaves = kBlock / 64;
constexpr int kW1 = 16, kW2 = 32, kW3 = 64;  // block widths (the paper's figure)
constexpr int kMaxK0 = 16;                   // d + f_d, zero-padded to 16
// The backward's per-entry record: h_0 (padded), h_1 and h_2 (the blocks'
// inputs), fp32, 256 bytes
constexpr int kRecH1 = kMaxK0, kRecH2 = kRecH1 + kW1, kRec = kRecH2 + kW2;
// LDS row of one output channel: 64 entries + 4 (16-byte aligned rows; the
// 16 lanes of a quarter-wave reading 16 bytes each then cover all 64 banks,
// and the MFMA output writes of the four lane quarters fall 16 banks apart)
constexpr int kYStride = 64 + 4;

// Per cloud (batch id), the group normalisation's sums (fp64) of the three
// blocks' inputs: block l's channel sums at kSum_l, sums of squares at kSq_l,
// then the row count; and the affines (fp32) the kernels apply: a at kAff_l,
// s at kAff_l + kAffW_l.  Block 1's input is padded to kMaxK0 channels.
constexpr int kSum0 = 0, kSq0 = 16, kSum1 = 32, kSq1 = 48, kSum2 = 64, kSq2 = 96, kCount = 128;
constexpr int kStatRow = 129;
constexpr int kAff0 = 0, kAff1 = 32, kAff2 = 64, kAffRow = 128;
// A cloud's batch id comes from its vertex's packed key (bits 48..63).  The
// per-cloud statistics cover batch ids below kGnClouds.
constexpr int kGnClouds = 64;
// Same-address fp64 atomics from many wavefronts serialise (about 0.1 us
// each, measured), so the statistics rows come in copies, each workgroup
// (batched) or wavefront (unbatched) adding to one copy, and the finalize
// adds the copies: kSpread copies of the one row of an unbatched lattice,
// kSpreadB copies of each of the kGnClouds rows of a batched one.
constexpr int kSpread = 64, kSpreadB = 16;
constexpr int kStatRows = kSpreadB * kGnClouds > kSpread ? kSpreadB * kGnClouds : kSpread;
__device__ __forceinline__ int64_t stat_row(int copy, int cloud, int batched) {
    return batched ? (int64_t)copy * kGnClouds + cloud : copy;
}
// A batched lattice's workgroups first add their rows in LDS (one row per
// cloud), then hand each row over once.

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
                                                         const uint64_t *__restrict__ vkeys, int batched,
                                                         int32_t *__restrict__ counters, int d,
                                                         int32_t *__restrict__ lvert, double *__restrict__ macc) {
    const int64_t V = counters[CNT_V];
    const int64_t nrows = counters[CNT_ROWS];
    const int64_t stride = (int64_t)gridDim.x * kBlock;
    int nclouds = 0;  // batched: 1 + the largest batch id among this thread's vertices
    for (int64_t v = (int64_t)blockIdx.x * kBlock + threadIdx.x; v < V; v += stride) {
        for (int i = 0; i < d; ++i) macc[v * d + i] = 0.0;
        if (batched) nclouds = max(nclouds, (int)(vkeys[v] >> 48) + 1);
        const int off = vinfo[2 * v], cnt = vinfo[2 * v + 1];
        if (cnt > kPart) continue;  // written by its parts below
        for (int e = off; e < off + cnt; ++e) lvert[e] = (int32_t)v;
    }
    if (batched) {
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) nclouds = max(nclouds, __shfl_xor(nclouds, o));
        if ((threadIdx.x & 63) == 0 && nclouds > 0) {
            atomicMax(counters + CNT_NB, nclouds);
            if (nclouds > kGnClouds) atomicOr(counters + CNT_STATUS, ST_CLOUDS);
        }
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

// Number of clouds whose statistics are kept: 1 for an unbatched lattice.
__device__ __forceinline__ int num_clouds(const int32_t *counters, int batched) {
    return batched ? min(counters[CNT_NB], kGnClouds) : 1;
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
        const int p = valid ? list_point(list[2 * e]) : 0;
        double acc[D];
#pragma unroll
        for (int i = 0; i < D; ++i) {
            const float pv = pos[(int64_t)p * D + i];  // unconditional (p = 0 past the end): the loads merge
            acc[i] = valid ? (double)pv : 0.0;
        }
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

// Without statistics the caller's (a, s) are the affines of the one row
// (cloud 0) the kernels read: block 1's zero-padded, then blocks 2 and 3.
__device__ __forceinline__ void affine_row(int64_t bid, int64_t nblk, const float *__restrict__ params, int k0,
                                           float *__restrict__ aff) {
    const int o1 = 2 * k0 + kW1 * k0 + kW1;  // block 2's a
    const int o2 = o1 + 2 * kW1 + kW2 * kW1 + kW2;  // block 3's a
    for (int64_t i = bid * kBlock + threadIdx.x; i < kAffRow; i += nblk * kBlock) {
        float x = 0.f;
        if (i < kAff1) {
            const int c = (int)i % kMaxK0;
            if (c < k0) x = params[(i < kMaxK0 ? 0 : k0) + c];
        } else if (i < kAff2) {
            x = params[o1 + (int)(i - kAff1)];  // a [16] then s [16]
        } else {
            x = params[o2 + (int)(i - kAff2)];  // a [32] then s [32]
        }
        aff[i] = x;
    }
}

// The statistics rows of the clouds present (or the copies of the one row),
// zeroed.
__device__ __forceinline__ void zero_stats(int64_t bid, int64_t nblk, const int32_t *__restrict__ counters,
                                           int batched, double *__restrict__ stats) {
    const int64_t n = (int64_t)kStatRows * kStatRow;
    for (int64_t i = bid * kBlock + threadIdx.x; i < n; i += nblk * kBlock) stats[i] = 0.0;
}

// After the local means: mu_v of the crossing lists, the key rows set to
// -inf, the parameters packed, and either the caller's affines copied (no
// statistics) or the statistics rows zeroed, in one launch (block ranges
// nb_mean, nb_rows, nb_pack, nb_gn).
__global__ __launch_bounds__(kBlock) void k_pointnet_prep(const int32_t *__restrict__ vinfo,
                                                          const double *__restrict__ macc, int d,
                                                          const int32_t *__restrict__ counters,
                                                          float *__restrict__ mu,
                                                          const int32_t *__restrict__ lvert,
                                                          unsigned int *__restrict__ keys,
                                                          const float *__restrict__ params, int k0,
                                                          float *__restrict__ padded, int gn, int batched,
                                                          double *__restrict__ stats, float *__restrict__ aff,
                                                          int nb_mean, int nb_rows, int nb_pack, int nb_gn) {
    const int b = blockIdx.x;
    if (b < nb_mean)
        mean_finish(b, nb_mean, vinfo, macc, d, counters, mu);
    else if (b < nb_mean + nb_rows)
        pointnet_rows<false>(b - nb_mean, nb_rows, lvert, vinfo, counters, 0, keys, nullptr);
    else if (b < nb_mean + nb_rows + nb_pack)
        pack_pointnet(b - nb_mean - nb_rows, nb_pack, params, k0, padded);
    else if (gn)
        zero_stats(b - nb_mean - nb_rows - nb_pack, nb_gn, counters, batched, stats);
    else
        affine_row(b - nb_mean - nb_rows - nb_pack, nb_gn, params, k0, aff);
}

// Sum x (and x^2) over the 16 lanes of a lane quarter (lanes with equal
// l / 16); every lane of the quarter gets the sums.
__device__ __forceinline__ double quarter_sum(double x) {
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) x += __shfl_xor(x, o);
    return x;
}

__device__ __forceinline__ double wave_sum(double x) {
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) x += __shfl_xor(x, o);
    return x;
}

// Group normalisation of block l's input (K channels in G groups of K / G):
// per cloud b and channel c, from the fp64 sums, mean and (biased) variance
// of c's group over the cloud's rows, then a = gamma_c / sqrt(var + eps) and
// s = beta_c - a mean, rounded once to fp32.  gamma and beta are the packed
// parameters' normalisation vectors.  Padded channels (c >= K) and absent
// clouds (no rows) get a = s = 0.  One wavefront per (cloud, channel), its
// lanes adding up the copies of the cloud's row.
__global__ __launch_bounds__(kBlock) void k_gn_finalize(const double *__restrict__ stats,
                                                        const float *__restrict__ P,
                                                        const int32_t *__restrict__ counters, int batched, int l,
                                                        int K, int G, float eps, float *__restrict__ aff) {
    const int KP = l == 2 ? kW2 : kMaxK0;
    const int sum_off = l == 0 ? kSum0 : (l == 1 ? kSum1 : kSum2);
    const int sq_off = l == 0 ? kSq0 : (l == 1 ? kSq1 : kSq2);
    const int aff_off = l == 0 ? kAff0 : (l == 1 ? kAff1 : kAff2);
    const int ga_off = l == 0 ? kA0 : (l == 1 ? kA1 : kA2);
    const int be_off = l == 0 ? kS0 : (l == 1 ? kS1 : kS2);
    const int lane = threadIdx.x & 63;
    const int64_t n = (int64_t)num_clouds(counters, batched) * KP;
    const int ncopy = batched ? kSpreadB : kSpread;
    const int gs = K / G;
    for (int64_t i = ((int64_t)blockIdx.x * kBlock + threadIdx.x) >> 6; i < n; i += (int64_t)gridDim.x * kWaves) {
        const int b = (int)(i / KP);
        const int c = (int)(i % KP);
        double rows = 0.0, sum = 0.0, sq = 0.0;
        if (lane < ncopy) {
            const double *st = stats + stat_row(lane, b, batched) * kStatRow;
            rows = st[kCount];
            if (c < K) {
                const int c0 = c / gs * gs;
                for (int j = c0; j < c0 + gs; ++j) {
                    sum += st[sum_off + j];
                    sq += st[sq_off + j];
                }
            }
        }
        rows = wave_sum(rows);
        sum = wave_sum(sum);
        sq = wave_sum(sq);
        float a = 0.f, s = 0.f;
        if (c < K && rows > 0.0) {
            const double cnt = rows * gs;
            const double mean = sum / cnt;
            double var = sq / cnt - mean * mean;
            var = var > 0.0 ? var : 0.0;
            const double ad = (double)P[ga_off + c] / sqrt(var + (double)eps);
            a = (float)ad;
            s = (float)((double)P[be_off + c] - ad * mean);
        }
        if (lane == 0) {
            aff[(int64_t)b * kAffRow + aff_off + c] = a;
            aff[(int64_t)b * kAffRow + aff_off + KP + c] = s;
        }
    }
}

// The cloud of entry e's vertex v: its batch id, 0 for an unbatched lattice.
// A batch id beyond the statistics' range (the call reports ST_CLOUDS) is
// clamped, so that every access stays in bounds.
__device__ __forceinline__ int cloud_of(const uint64_t *__restrict__ vkeys, int batched, int v) {
    return batched ? min((int)(vkeys[v] >> 48), kGnClouds - 1) : 0;
}

// Per cloud, the row count and the sums of h_0 = [g_p - mu_v ; f_p] and of
// its squares per channel.  One lane per entry; each wavefront takes one
// contiguous range of chunks, so that its cloud changes only at the clouds'
// boundaries, and adds up its rows in registers while they stay in one
// cloud.  Unbatched, the sums go to the wavefront's copy of the one row at
// the end.  Batched, they go (and the rows of a chunk that spans several
// clouds go one by one) to the workgroup's LDS row of the cloud, and the
// workgroup hands its rows over at the end.
template <int D>
__global__ __launch_bounds__(kBlock) void k_gn_stats0(const int32_t *__restrict__ list,
                                                      const int32_t *__restrict__ lvert,
                                                      const uint64_t *__restrict__ vkeys, int batched,
                                                      const float *__restrict__ pos, const float *__restrict__ feat,
                                                      int f_d, const float *__restrict__ mu,
                                                      const int32_t *__restrict__ counters,
                                                      double *__restrict__ stats) {
    constexpr int ROW = 2 * kMaxK0 + 1;  // sums, sums of squares, count
    __shared__ double tbl[kGnClouds * ROW];
    const int64_t E = counters[CNT_E];
    const int lane = threadIdx.x & 63;
    const int k0 = D + f_d;
    const int nb = num_clouds(counters, batched);
    if (batched) {
        for (int i = threadIdx.x; i < nb * ROW; i += kBlock) tbl[i] = 0.0;
        __syncthreads();
    }
    const int64_t nwaves = (int64_t)gridDim.x * kWaves;
    const int64_t wave = ((int64_t)blockIdx.x * kBlock + threadIdx.x) >> 6;
    const int64_t nch = (E + 63) / 64, per = (nch + nwaves - 1) / nwaves;
    const int64_t c_lo = wave * per, c_hi = c_lo + per < nch ? c_lo + per : nch;
    double s[kMaxK0], q[kMaxK0], cnt = 0.0;
#pragma unroll
    for (int i = 0; i < kMaxK0; ++i) s[i] = q[i] = 0.0;
    int held = -1;  // the cloud whose rows s, q, cnt hold (wave-uniform)
    auto flush = [&]() {
        if (held < 0) return;
        const double c = wave_sum(cnt);
#pragma unroll
        for (int i = 0; i < kMaxK0; ++i) {
            s[i] = wave_sum(s[i]);
            q[i] = wave_sum(q[i]);
        }
        if (lane == 0) {
            if (batched) {
                double *row = tbl + held * ROW;  // LDS
                atomicAdd(row + 2 * kMaxK0, c);
                for (int i = 0; i < k0; ++i) {
                    atomicAdd(row + i, s[i]);
                    atomicAdd(row + kMaxK0 + i, q[i]);
                }
            } else {
                double *st = stats + stat_row((int)(wave % kSpread), 0, 0) * kStatRow;
                atomicAdd(st + kCount, c);
                for (int i = 0; i < k0; ++i) {
                    atomicAdd(st + kSum0 + i, s[i]);
                    atomicAdd(st + kSq0 + i, q[i]);
                }
            }
        }
#pragma unroll
        for (int i = 0; i < kMaxK0; ++i) s[i] = q[i] = 0.0;
        cnt = 0.0;
        held = -1;
    };
    for (int64_t c = c_lo; c < c_hi; ++c) {
        const int64_t e = c * 64 + lane;
        const bool valid = e < E;
        const int v = valid ? lvert[e] : 0;
        const int p = valid ? list_point(list[2 * e]) : 0;
        const int b = valid ? cloud_of(vkeys, batched, v) : -1;
        float x[kMaxK0];
#pragma unroll
        for (int i = 0; i < kMaxK0; ++i) {
            float t = 0.f;
            if (i < D) {
                // unconditional (p = v = 0 past the end), so that the D
                // adjacent loads merge into one
                const float pv = pos[(int64_t)p * D + i], mv = mu[(int64_t)v * D + i];
                t = valid ? pv - mv : 0.f;
            } else if (valid && i < k0) {
                t = feat[(int64_t)p * f_d + (i - D)];
            }
            x[i] = t;
        }
        const int bref = __builtin_amdgcn_readfirstlane(b);  // lane 0 is valid in every chunk
        const bool uniform = __ballot(valid && b != bref) == 0ull;
        if (uniform) {
            if (bref != held) {
                flush();
                held = bref;
            }
            cnt += valid ? 1.0 : 0.0;
#pragma unroll
            for (int i = 0; i < kMaxK0; ++i) {
                const double t = (double)x[i];
                s[i] += t;
                q[i] += t * t;
            }
        } else if (valid) {  // only batched lattices have chunks that span clouds
            double *row = tbl + b * ROW;
            atomicAdd(row + 2 * kMaxK0, 1.0);
            for (int i = 0; i < k0; ++i) {
                const double t = (double)x[i];
                atomicAdd(row + i, t);
                atomicAdd(row + kMaxK0 + i, t * t);
            }
        }
    }
    flush();
    if (batched) {
        __syncthreads();
        const int copy = (int)(blockIdx.x % kSpreadB);
        for (int i = threadIdx.x; i < nb * ROW; i += kBlock) {
            const int b = i / ROW, j = i % ROW;
            const double x = tbl[i];
            if (x == 0.0) continue;
            const int at = j == 2 * kMaxK0 ? kCount : (j < kMaxK0 ? kSum0 + j : kSq0 + (j - kMaxK0));
            atomicAdd(stats + stat_row(copy, b, 1) * kStatRow + at, x);
        }
    }
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
// lane stages its own row).  Each wavefront loops over its own chunks
// (wavefront-level synchronisation only).
//   MODE 1: block 1 only; the sums of h_1 and h_1^2 per cloud and channel.
//   MODE 2: blocks 1 and 2; the sums of h_2 and h_2^2.
//   MODE 3: all three blocks; the outputs go to LDS channel-major for the
//           per-run max (see the file comment).
// The normalisations are the per-cloud affines aff[cloud][..] (one row
// when the lattice is unbatched or the caller gave the affines).  A chunk
// whose entries all belong to one cloud (every chunk of an unbatched
// lattice) uses that cloud's affines, kept in registers while the cloud
// stays the same; a chunk that spans clouds loads each entry's own.
template <int MODE, bool OUT_BF16>
__global__ __launch_bounds__(kBlock, 2) void k_pointnet(const int32_t *__restrict__ list,
                                                     const int32_t *__restrict__ lvert,
                                                     const int32_t *__restrict__ vinfo,
                                                     const uint64_t *__restrict__ vkeys, int batched,
                                                     const float *__restrict__ pos, const float *__restrict__ feat,
                                                     int d, int f_d, const float *__restrict__ P,
                                                     const float *__restrict__ aff,
                                                     const float *__restrict__ mu,
                                                     const int32_t *__restrict__ counters,
                                                     double *__restrict__ stats,
                                                     unsigned int *__restrict__ keys, void *__restrict__ out,
                                                     float *__restrict__ rec, uint64_t *__restrict__ routed,
                                                     int32_t *__restrict__ win, uint2 *__restrict__ wslot) {
    // MODE 3, 4: outputs [64 channels][64 entries], first the staged inputs;
    // MODE 1, 2: the staged inputs only
    constexpr int kYWave = MODE >= 3 ? kW3 * kYStride : 64 * (kMaxK0 + 1);
    __shared__ __attribute__((aligned(16))) float ysh[kWaves][kYWave];
    // MODE 1, 2 on a batched lattice: the workgroup's sums (then sums of
    // squares) of the block's output per cloud
    constexpr int KS = MODE == 1 ? kW1 : kW2;
    __shared__ double gtbl[MODE < 3 ? kGnClouds * 2 * KS : 1];

    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int q = lane >> 4, j16 = lane & 15;
    float *Y = ysh[w];
    const int k0 = d + f_d;

    // weight fragments (A operands) and biases of this lane
    float wa1[4], bias1[4];
    float wa2[2][4], bias2[2][4];
    float wa3[4][8], bb3[4][4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        wa1[t] = P[kWt0 + j16 * kMaxK0 + 4 * t + q];  // block 1: K = 4 t + q (the staged input order)
        bias1[t] = P[kB0 + 4 * q + t];                 // block 1 output channel in register t
    }
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            wa2[mt][t] = P[kWt1 + (16 * mt + j16) * kW1 + 4 * q + t];  // block 2: K = 4 q + t
            bias2[mt][t] = P[kB1 + 16 * mt + 4 * q + t];
        }
#pragma unroll
    for (int mt = 0; mt < 4; ++mt) {
#pragma unroll
        for (int t = 0; t < 8; ++t)  // block 3: K = 16 (t / 4) + 4 q + t % 4
            wa3[mt][t] = P[kWt2 + (16 * mt + j16) * kW2 + 16 * (t / 4) + 4 * q + (t % 4)];
#pragma unroll
        for (int r = 0; r < 4; ++r) bb3[mt][r] = P[kB2 + 16 * mt + 4 * q + r];
    }

    // The normalisations of one cloud, in this lane's layout: the staged
    // input's (channel i of the lane's own entry) and, for the MFMA outputs
    // in register t of row tile mt, channel 4 q + t (+16 mt).  The next
    // block's bias is folded in: a (h + b) + s = a h + (a b + s).
    struct Aff {
        float a0[kMaxK0], s0[kMaxK0];
        float a1[4], s1[4];
        float a2[2][4], s2[2][4];
    };
    auto load_stage = [&](int b, float *a0, float *s0) {
        const float *A = aff + (int64_t)b * kAffRow;
#pragma unroll
        for (int i = 0; i < kMaxK0; ++i) {
            a0[i] = A[kAff0 + i];
            s0[i] = A[kAff0 + kMaxK0 + i];
        }
    };
    auto load_inner = [&](int b, float *a1, float *s1, float (*a2)[4], float (*s2)[4]) {
        const float *A = aff + (int64_t)b * kAffRow;
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            const int c = 4 * q + t;
            a1[t] = A[kAff1 + c];
            s1[t] = fmaf(a1[t], bias1[t], A[kAff1 + kW1 + c]);
        }
        if (MODE >= 3) {
#pragma unroll
            for (int mt = 0; mt < 2; ++mt)
#pragma unroll
                for (int t = 0; t < 4; ++t) {
                    const int c = 16 * mt + 4 * q + t;
                    a2[mt][t] = A[kAff2 + c];
                    s2[mt][t] = fmaf(a2[mt][t], bias2[mt][t], A[kAff2 + kW2 + c]);
                }
        }
    };
    Aff U;  // the affines of cloud `held` (wave-uniform)
    int held = -1;

    const int64_t E = counters[CNT_E];
    const int64_t nwaves = (int64_t)gridDim.x * kWaves;
    const int64_t wave = ((int64_t)blockIdx.x * kBlock + threadIdx.x) >> 6;
    // This wavefront's chunks: strided over the grid for the final pass; one
    // contiguous range for the statistics passes, so that a wavefront's
    // cloud changes only at the clouds' boundaries.
    const int64_t nch = (E + 63) / 64, per = (nch + nwaves - 1) / nwaves;
    const int64_t c_first = MODE >= 3 ? wave : wave * per;
    const int64_t c_end = MODE >= 3 ? nch : (c_first + per < nch ? c_first + per : nch);
    const int64_t step = MODE >= 3 ? nwaves : 1;
    // statistics of this lane's channels of the block's output (MODE 1:
    // channel 4 q + t; MODE 2: 16 mt + 4 q + t) over the rows of cloud
    // `sheld`, handed over when the cloud changes and at the end
    constexpr int NS = MODE == 1 ? 4 : (MODE == 2 ? 8 : 1);
    double ss[NS], sq[NS];
#pragma unroll
    for (int i = 0; i < NS; ++i) ss[i] = sq[i] = 0.0;
    int sheld = -1;
    auto chan = [&](int i) { return MODE == 1 ? 4 * q + i : 16 * (i / 4) + 4 * q + (i % 4); };
    const int so = MODE == 1 ? kSum1 : kSum2, qo = MODE == 1 ? kSq1 : kSq2;
    if (MODE < 3 && batched) {
        for (int i = threadIdx.x; i < num_clouds(counters, batched) * 2 * KS; i += kBlock) gtbl[i] = 0.0;
        __syncthreads();
    }
    auto flush = [&]() {
        if (MODE >= 3 || sheld < 0) return;
#pragma unroll
        for (int i = 0; i < NS; ++i) {
            ss[i] = quarter_sum(ss[i]);
            sq[i] = quarter_sum(sq[i]);
        }
        if (j16 == 0) {
            if (batched) {
                double *row = gtbl + sheld * 2 * KS;  // LDS
#pragma unroll
                for (int i = 0; i < NS; ++i) {
                    atomicAdd(row + chan(i), ss[i]);
                    atomicAdd(row + KS + chan(i), sq[i]);
                }
            } else {
                double *st = stats + stat_row((int)(wave % kSpread), 0, 0) * kStatRow;
#pragma unroll
                for (int i = 0; i < NS; ++i) {
                    atomicAdd(st + so + chan(i), ss[i]);
                    atomicAdd(st + qo + chan(i), sq[i]);
                }
            }
        }
#pragma unroll
        for (int i = 0; i < NS; ++i) ss[i] = sq[i] = 0.0;
        sheld = -1;
    };

    // Software pipeline over this wavefront's chunks: the entry's vertex and
    // point (level 1) are loaded two chunks ahead, the vertex's list header,
    // cloud, the point's position and features and the vertex's mean (level
    // 2, which need level 1) one chunk ahead, so that a chunk's MFMAs never
    // wait on its own gathers.
    const bool pos4 = d == 4 && ((reinterpret_cast<uintptr_t>(pos) | reinterpret_cast<uintptr_t>(mu)) & 15) == 0;
    struct Rows {
        int v, p;             // level 1
        int off, cnt, b;      // level 2
        float x[kMaxK0];      // h_0 (level 2)
    };
    auto level1 = [&](int64_t chk, Rows &R) {
        const int64_t e = chk * 64 + lane;
        const bool valid = e < E;
        R.v = valid ? lvert[e] : -1;
        R.p = valid ? list_point(list[2 * e]) : 0;
    };
    auto level2 = [&](Rows &R) {
        const bool valid = R.v >= 0;
        R.off = valid ? vinfo[2 * R.v] : 0;
        R.cnt = valid ? vinfo[2 * R.v + 1] : 0;
        R.b = valid ? cloud_of(vkeys, batched, R.v) : -1;
        if (pos4) {
            // d = 4 with 16-byte aligned rows: the position and the mean as
            // one 16-byte load each
            const float4 pp = valid ? reinterpret_cast<const float4 *>(pos)[R.p] : make_float4(0.f, 0.f, 0.f, 0.f);
            const float4 mm = valid ? reinterpret_cast<const float4 *>(mu)[R.v] : make_float4(0.f, 0.f, 0.f, 0.f);
            R.x[0] = pp.x - mm.x;
            R.x[1] = pp.y - mm.y;
            R.x[2] = pp.z - mm.z;
            R.x[3] = pp.w - mm.w;
#pragma unroll
            for (int i = 4; i < kMaxK0; ++i) R.x[i] = valid && i < k0 ? feat[(int64_t)R.p * f_d + (i - 4)] : 0.f;
        } else if (d == 3) {
            // d = 3: three adjacent 4-byte loads each (unconditional, so that
            // they merge into one 12-byte load)
            const int64_t p3 = (int64_t)(valid ? R.p : 0) * 3, v3 = (int64_t)(valid ? R.v : 0) * 3;
            const float p0 = pos[p3], p1 = pos[p3 + 1], p2 = pos[p3 + 2];
            const float m0 = mu[v3], m1 = mu[v3 + 1], m2 = mu[v3 + 2];
            R.x[0] = valid ? p0 - m0 : 0.f;
            R.x[1] = valid ? p1 - m1 : 0.f;
            R.x[2] = valid ? p2 - m2 : 0.f;
#pragma unroll
            for (int i = 3; i < kMaxK0; ++i) R.x[i] = valid && i < k0 ? feat[(int64_t)R.p * f_d + (i - 3)] : 0.f;
        } else {
#pragma unroll
            for (int i = 0; i < kMaxK0; ++i) {
                float x = 0.f;
                if (valid && i < d) x = pos[(int64_t)R.p * d + i] - mu[(int64_t)R.v * d + i];
                else if (valid && i < k0) x = feat[(int64_t)R.p * f_d + (i - d)];
                R.x[i] = x;
            }
        }
    };
    int64_t ch = c_first;
    Rows cur, nxt;
    int v2 = -1, p2 = 0;
    if (ch < c_end) {
        level1(ch, cur);
        level2(cur);
        level1(ch + step, nxt);
    }
    for (; ch < c_end; ch += step) {
        // issue the next chunk's level 2 and the one after's level 1 (past
        // this wavefront's range they are loaded and not used)
        {
            Rows tmp;
            tmp.v = nxt.v;
            tmp.p = nxt.p;
            const int64_t e2 = (ch + 2 * step) * 64 + lane;
            v2 = e2 < E ? lvert[e2] : -1;
            p2 = e2 < E ? list_point(list[2 * e2]) : 0;
            level2(tmp);
            nxt = tmp;
        }
        const int64_t chunk0 = ch * 64;
        const int v = cur.v;
        const bool valid = v >= 0;
        // the chunk's cloud: lane 0's (every chunk's first entry is valid),
        // and whether every entry shares it
        const int bref = __builtin_amdgcn_readfirstlane(cur.b);
        const bool uniform = __ballot(valid && cur.b != bref) == 0ull;
        if (uniform && bref != held) {
            load_stage(bref, U.a0, U.s0);
            load_inner(bref, U.a1, U.s1, U.a2, U.s2);
            held = bref;
        }
        if (MODE < 3 && (!uniform || bref != sheld)) {
            flush();
            if (uniform) sheld = bref;
        }
        // MODE 4: the entry's record starts with h_0, and its routing mask
        // is cleared (the backward's argmax sets the masks of the winners)
        if (MODE == 4 && valid) {
            float *R = rec + (chunk0 + lane) * kRec;
#pragma unroll
            for (int i = 0; i < kMaxK0; i += 4)
                *reinterpret_cast<float4 *>(R + i) = make_float4(cur.x[i], cur.x[i + 1], cur.x[i + 2], cur.x[i + 3]);
            routed[chunk0 + lane] = 0ull;
        }
        // run flags: 1 first entry of a run, 2 last, 4 the run is the vertex's whole list
        int flags = 0, dest = -1;
        if (MODE >= 3) {
            const int vprev = __shfl_up(v, 1);
            const int vnext = __shfl_down(v, 1);
            if (valid) {
                if (lane == 0 || vprev != v) flags |= 1;
                if (lane == 63 || vnext != v) flags |= 2;
                if (cur.off >= chunk0 && cur.off + cur.cnt <= chunk0 + 64) flags |= 4;
            }
            // destination of the run: the output row, or the key row of the
            // chunk where the vertex's list starts
            dest = (flags & 4) ? v : (valid ? (int)(cur.off >> 6) : -1);
        }

        // r_0 = relu(a_0 h_0 + s_0), h_0 = [g_p - mu_v ; f_p] zero-padded, staged in LDS
        {
            float a0[kMaxK0], s0[kMaxK0];
            if (uniform) {
#pragma unroll
                for (int i = 0; i < kMaxK0; ++i) {
                    a0[i] = U.a0[i];
                    s0[i] = U.s0[i];
                }
            } else {
                load_stage(valid ? cur.b : 0, a0, s0);
            }
#pragma unroll
            for (int i = 0; i < kMaxK0; ++i) Y[lane * (kMaxK0 + 1) + i] = relu(fmaf(a0[i], cur.x[i], s0[i]));
        }
        wave_sync();
        float b1[4][4];  // B operands of block 1: entry 16 nt + j16, K = 4 t + q
#pragma unroll
        for (int nt = 0; nt < 4; ++nt)
#pragma unroll
            for (int t = 0; t < 4; ++t) b1[nt][t] = Y[(16 * nt + j16) * (kMaxK0 + 1) + 4 * t + q];
        wave_sync();

#pragma unroll
        for (int nt = 0; nt < 4; ++nt) {
            // this lane's entry in the tile: its cloud and validity
            const int ebv = __shfl(valid ? cur.b : -1, 16 * nt + j16);
            float a1[4], s1[4], a2[2][4], s2[2][4];
            if (uniform) {
#pragma unroll
                for (int t = 0; t < 4; ++t) {
                    a1[t] = U.a1[t];
                    s1[t] = U.s1[t];
                    a2[0][t] = U.a2[0][t];
                    s2[0][t] = U.s2[0][t];
                    a2[1][t] = U.a2[1][t];
                    s2[1][t] = U.s2[1][t];
                }
            } else if (MODE >= 2) {
                load_inner(ebv >= 0 ? ebv : 0, a1, s1, a2, s2);
            }
            f32x4_t d1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int t = 0; t < 4; ++t) d1 = mfma16(wa1[t], b1[nt][t], d1);
            if (MODE == 1) {
#pragma unroll
                for (int t = 0; t < 4; ++t) {
                    const double h = ebv >= 0 ? (double)(d1[t] + bias1[t]) : 0.0;
                    if (uniform) {
                        ss[t] += h;
                        sq[t] += h * h;
                    } else if (ebv >= 0) {  // only batched lattices have chunks that span clouds
                        double *row = gtbl + ebv * 2 * KS;
                        atomicAdd(row + chan(t), h);
                        atomicAdd(row + KS + chan(t), h * h);
                    }
                }
                continue;
            }
            float r1[4];
#pragma unroll
            for (int t = 0; t < 4; ++t) r1[t] = relu(fmaf(a1[t], d1[t], s1[t]));
            f32x4_t d2[2];
#pragma unroll
            for (int mt = 0; mt < 2; ++mt) {
                d2[mt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int t = 0; t < 4; ++t) d2[mt] = mfma16(wa2[mt][t], r1[t], d2[mt]);
            }
            if (MODE == 2) {
#pragma unroll
                for (int i = 0; i < 8; ++i) {
                    const double h = ebv >= 0 ? (double)(d2[i / 4][i % 4] + bias2[i / 4][i % 4]) : 0.0;
                    if (uniform) {
                        ss[i] += h;
                        sq[i] += h * h;
                    } else if (ebv >= 0) {
                        double *row = gtbl + ebv * 2 * KS;
                        atomicAdd(row + chan(i), h);
                        atomicAdd(row + KS + chan(i), h * h);
                    }
                }
                continue;
            }
            float r2[8];
#pragma unroll
            for (int t = 0; t < 8; ++t)
                r2[t] = relu(fmaf(a2[t / 4][t % 4], d2[t / 4][t % 4], s2[t / 4][t % 4]));
            // MODE 4: this lane's four channels of h_1 and h_2 of entry
            // 16 nt + j16 go to its record
            float *R = MODE == 4 ? rec + (chunk0 + 16 * nt + j16) * kRec : nullptr;
            if (MODE == 4 && ebv >= 0) {
                *reinterpret_cast<float4 *>(R + kRecH1 + 4 * q) =
                    make_float4(d1[0] + bias1[0], d1[1] + bias1[1], d1[2] + bias1[2], d1[3] + bias1[3]);
#pragma unroll
                for (int mt = 0; mt < 2; ++mt)
                    *reinterpret_cast<float4 *>(R + kRecH2 + 16 * mt + 4 * q) =
                        make_float4(d2[mt][0] + bias2[mt][0], d2[mt][1] + bias2[mt][1], d2[mt][2] + bias2[mt][2],
                                    d2[mt][3] + bias2[mt][3]);
            }
#pragma unroll
            for (int mt = 0; mt < 4; ++mt) {
                f32x4_t d3 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int t = 0; t < 8; ++t) d3 = mfma16(wa3[mt][t], r2[t], d3);
#pragma unroll
                for (int r = 0; r < 4; ++r) Y[(16 * mt + 4 * q + r) * kYStride + 16 * nt + j16] = d3[r] + bb3[mt][r];
            }
        }

        if (MODE == 3) {
            wave_sync();
            // lane c: running max of channel c over each run of the wavefront's
            // entries, four entries per LDS read; an entry's run flags and
            // destination come from its lane (readlane: scalar values, so the
            // store at a run's end is a uniform branch)
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
        if (MODE == 4) {
            wave_sync();
            // lane c: the first maximum of channel c over each run of the
            // wavefront's entries (the values the forward's max takes, in
            // entry order), kept at the end of the run: the winning entry of
            // a list that lies within this chunk; for a list that crosses a
            // chunk boundary, the run's (value, entry) in slot 0 of the chunk
            // (the run that holds the chunk's first entry) or slot 1 (the run
            // that holds its last), which the argmax combines in chunk order
            const int c = lane;
            float mx = 0.f;
            int be = 0, r0 = 0;
#pragma unroll
            for (int j4 = 0; j4 < 16; ++j4) {
                const f32x4_t y4 = *reinterpret_cast<const f32x4_t *>(Y + c * kYStride + 4 * j4);
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int jj = 4 * j4 + i;
                    const int fj = __builtin_amdgcn_readlane(flags, jj);
                    if (fj & 1) r0 = jj;
                    if ((fj & 1) || y4[i] > mx) {
                        mx = y4[i];
                        be = jj;
                    }
                    if (fj & 2) {
                        if (fj & 4)
                            win[(int64_t)__builtin_amdgcn_readlane(dest, jj) * kW3 + c] = (int32_t)(chunk0 + be);
                        else
                            wslot[(ch * 2 + (r0 == 0 ? 0 : 1)) * kW3 + c] =
                                make_uint2(__float_as_uint(mx), (uint32_t)(chunk0 + be));
                    }
                }
            }
        }
        wave_sync();
        cur = nxt;
        nxt.v = v2;
        nxt.p = p2;
    }
    flush();
    if (MODE < 3 && batched) {
        __syncthreads();
        const int copy = (int)(blockIdx.x % kSpreadB);
        for (int i = threadIdx.x; i < num_clouds(counters, batched) * 2 * KS; i += kBlock) {
            const int b = i / (2 * KS), j = i % (2 * KS);
            const double x = gtbl[i];
            if (x != 0.0) atomicAdd(stats + stat_row(copy, b, 1) * kStatRow + (j < KS ? so + j : qo + (j - KS)), x);
        }
    }
}

// ---------------------------------------------------------------------------
// Backward of the PointNet blocks: the gradients of every block's parameters
// (gamma and beta, or a and s; W; b) given g = dL/dx [V][64].  The positions
// and features are the network's raw inputs and get none.  With the forward
// run first (its statistics, affines, local means and entry-to-vertex map),
// per entry e of vertex v (one row):
//   k_dpn_norm     per cloud and block, each input channel's group mean and
//                  1 / sqrt(var + eps) from the fp64 sums (mean 0, 1 for the
//                  fixed affine)
//   k_pointnet<4>  the forward's MFMA pass once more: the record of e (block
//                  inputs h0 (padded), h1, h2, fp32) and, per vertex and
//                  channel c, the entry whose h3[c] is largest (the first in
//                  list order), found over each run of a wavefront's entries
//                  as the forward's max is (the values its max took)
//   k_dpn_argmax   one wavefront per vertex, lane = channel c: the winning
//                  row (a list that crosses chunks: its runs' winners combined
//                  in chunk order) receives g[v][c]; dW3[c][.] += g r3 and
//                  db3[c] += g of that row; per entry the mask of the channels
//                  it receives
//   k_dpn_back<S>  one wavefront per workgroup, a lane per entry: back through
//                  block 3 (S = 3: dhn3 from the routed channels, stored per
//                  entry; dgamma3, dbeta3 and the group sums of gamma dhn and
//                  gamma dhn xhat), block 2 (S = 2: needs block 3's group
//                  means; dhn2 stored per entry; dW2, db2, dgamma2, dbeta2,
//                  block 2's group sums) or block 1 (S = 1: dW1, db1, dgamma1,
//                  dbeta1).  A group normalisation's input gradient is rstd
//                  (gn - mean(gn) - xhat mean(gn xhat)), gn = gamma dhn, the
//                  means over the cloud's rows and the group's channels.
// Sums over entries, per chunk of 64 entries: the entries' vectors are staged
// in the wavefront's LDS; lane c adds column c over them, in entry order, into
// a register kept over the wavefront's chunks (the per-channel sums); the
// weight gradients dW = sum_e dh_e r_e^T run on fp32 MFMA 32x32x2 (two entries
// a step) into accumulators kept the same way.  A group sum is a gamma-weighted
// sum of per-channel sums: with one cloud it is formed from those at the end;
// with several, lane (group, part) adds each entry to its cloud's slot of an
// LDS table, in entry order.  Each wavefront writes one partial row; the rows
// are added in a fixed order (rowsum): the gradients do not depend on
// scheduling.  Lanes past the last entry add zeros: with group normalisation
// an input gradient has mean terms even where no output gradient reaches the
// row, so such lanes zero theirs explicitly.
constexpr int kNrmRow = 3 * 2 * 32;              // per cloud: (mean, rstd) per block and input channel
constexpr int kPArg = kW3 * kW2 + kW3;                           // per wavefront: dW3, db3
// Partial rows of the passes: S = 3 dgamma3 [32], dbeta3 [32]; S = 2 dW2
// [32][16], db2 [32], dgamma2 [16], dbeta2 [16]; S = 1 dW1 [16][16], db1
// [16], dgamma1 [16], dbeta1 [16]; then (S = 3, 2) the group sums, slot
// (cloud K + group) 2 + part, of one cloud or (batched) of kGnClouds.
constexpr int kPB3Base = 2 * kW2, kPB2Base = kW2 * kW1 + kW2 + 2 * kW1;
constexpr int kPB3 = kPB3Base + kGnClouds * kW2 * 2;
constexpr int kPB2 = kPB2Base + kGnClouds * kW1 * 2;
constexpr int kPB1 = kW1 * kMaxK0 + kW1 + 2 * kMaxK0;
__host__ __device__ inline int pb_len(int S, int batched) {
    const int nc = batched ? kGnClouds : 1;
    return S == 3 ? kPB3Base + nc * kW2 * 2 : (S == 2 ? kPB2Base + nc * kW1 * 2 : kPB1);
}
// staged floats per entry (64-entry chunks); an odd pitch puts a lane's own
// row writes and the column reads on 64 different banks
constexpr int kStg = 81;
constexpr int kSparseBits = 24;  // pass 3 visits only the routed channels when no entry has more

typedef float f32x16_t __attribute__((ext_vector_type(16)));

// Block l's input width (l = 0, 1, 2) and its padded width.
__host__ __device__ __forceinline__ int in_width(int l, int k0) { return l == 0 ? k0 : (l == 1 ? kW1 : kW2); }
__host__ __device__ __forceinline__ int in_padded(int l) { return l == 2 ? kW2 : kMaxK0; }

__global__ __launch_bounds__(kBlock) void k_dpn_norm(const double *__restrict__ stats,
                                                     const int32_t *__restrict__ counters, int batched, int use_gn,
                                                     int k0, int G0, int G1, int G2, float eps,
                                                     float *__restrict__ nrm, double *__restrict__ rows_out) {
    const int lane = threadIdx.x & 63;
    const int64_t n = (int64_t)num_clouds(counters, batched) * 3 * 32;
    const int ncopy = batched ? kSpreadB : kSpread;
    for (int64_t i = ((int64_t)blockIdx.x * kBlock + threadIdx.x) >> 6; i < n; i += (int64_t)gridDim.x * kWaves) {
        const int b = (int)(i / 96);
        const int l = (int)(i % 96) / 32;
        const int c = (int)(i % 32);
        const int K = in_width(l, k0);
        const int G = l == 0 ? G0 : (l == 1 ? G1 : G2);
        float mean = 0.f, rstd = 1.f;
        double rows = 0.0;
        if (use_gn) {
            const int sum_off = l == 0 ? kSum0 : (l == 1 ? kSum1 : kSum2);
            const int sq_off = l == 0 ? kSq0 : (l == 1 ? kSq1 : kSq2);
            const int gs = K / G;
            double sum = 0.0, sq = 0.0;
            if (lane < ncopy) {
                const double *st = stats + stat_row(lane, b, batched) * kStatRow;
                rows = st[kCount];
                if (c < K) {
                    const int c0 = c / gs * gs;
                    for (int j = c0; j < c0 + gs; ++j) {
                        sum += st[sum_off + j];
                        sq += st[sq_off + j];
                    }
                }
            }
            rows = wave_sum(rows);
            sum = wave_sum(sum);
            sq = wave_sum(sq);
            if (c < K && rows > 0.0) {
                const double cnt = rows * gs;
                const double m = sum / cnt;
                double var = sq / cnt - m * m;
                var = var > 0.0 ? var : 0.0;
                mean = (float)m;
                rstd = (float)(1.0 / sqrt(var + (double)eps));
            }
        }
        if (lane == 0) {
            nrm[(int64_t)b * kNrmRow + l * 64 + 2 * c] = mean;
            nrm[(int64_t)b * kNrmRow + l * 64 + 2 * c + 1] = rstd;
            if (l == 0 && c == 0) rows_out[b] = rows;
        }
    }
}

// Stage the padded parameters in LDS.
__device__ __forceinline__ void load_params(const float *__restrict__ P, float *Ps) {
    for (int i = threadIdx.x; i < kPadded; i += kBlock) Ps[i] = P[i];
    __syncthreads();
}

__global__ __launch_bounds__(kBlock) void k_dpn_argmax(const int32_t *__restrict__ vinfo,
                                                       const uint64_t *__restrict__ vkeys, int batched,
                                                       const float *__restrict__ aff, const float *__restrict__ rec,
                                                       const int32_t *__restrict__ win,
                                                       const uint2 *__restrict__ wslot,
                                                       const float *__restrict__ grad_out,
                                                       const int32_t *__restrict__ counters,
                                                       uint64_t *__restrict__ routed, float *__restrict__ part) {
    const int lane = threadIdx.x & 63;  // output channel c
    const int64_t V = counters[CNT_V];
    const int64_t wave = ((int64_t)blockIdx.x * kBlock + threadIdx.x) >> 6;
    const int64_t nwaves = ((int64_t)gridDim.x * kBlock) >> 6;
    float dw[kW2], db = 0.f;
#pragma unroll
    for (int j = 0; j < kW2; ++j) dw[j] = 0.f;
    for (int64_t v = wave; v < V; v += nwaves) {
        const int64_t off = vinfo[2 * v];
        const int cnt = vinfo[2 * v + 1];
        // the winning entry of channel c (the first maximum in list order):
        // recorded by the records pass for a list within one chunk, else
        // the runs' slots combined in chunk order
        const int64_t j0 = off >> 6, j1 = (off + cnt - 1) >> 6;
        int be;
        if (j0 == j1) {
            be = win[v * kW3 + lane];
        } else {
            float best = 0.f;
            be = (int)off;
            for (int64_t j = j0; j <= j1; ++j) {
                const int sl = (j == j0 && (off & 63) != 0) ? 1 : 0;
                const uint2 r = wslot[(j * 2 + sl) * kW3 + lane];
                const float x = __uint_as_float(r.x);
                if (j == j0 || x > best) {
                    best = x;
                    be = (int)r.y;
                }
            }
        }
        // the mask of each winning entry (the others were zeroed with their
        // records): one store per distinct winner, by its first lane
        uint64_t todo = ~0ull;
        while (todo) {
            const int leader = __builtin_ctzll(todo);
            const int w = __shfl(be, leader);
            const uint64_t mk = __ballot(be == w);
            if (lane == leader) routed[w] = mk;
            todo &= ~mk;
        }
        const float g = grad_out[v * kW3 + lane];
        db += g;
        const float *A = aff + (int64_t)cloud_of(vkeys, batched, (int)v) * kAffRow;
        const float *R = rec + (int64_t)be * kRec + kRecH2;
#pragma unroll
        for (int j = 0; j < kW2; ++j) dw[j] = fmaf(g, relu(fmaf(A[kAff2 + j], R[j], A[kAff2 + kW2 + j])), dw[j]);
    }
    float *out = part + wave * kPArg;
#pragma unroll
    for (int j = 0; j < kW2; ++j) out[lane * kW2 + j] = dw[j];
    out[kW3 * kW2 + lane] = db;
}

// One backward pass (see above).  din: the previous pass's stored per-entry
// gradient (S = 2: dhn3 [E][32], S = 1: dhn2 [E][16]); dout: this pass's
// (S = 3: dhn3, S = 2: dhn2).  One wavefront per workgroup.
template <int S, bool BATCHED>
__global__ __launch_bounds__(64) void k_dpn_back(const int32_t *__restrict__ lvert,
                                                 const uint64_t *__restrict__ vkeys, int batched, int use_gn, int G1,
                                                 int G2, const float *__restrict__ P, const float *__restrict__ aff,
                                                 const float *__restrict__ nrm, const float *__restrict__ gm,
                                                 const float *__restrict__ rec, const uint64_t *__restrict__ routed,
                                                 const float *__restrict__ grad_out, const float *__restrict__ din,
                                                 float *__restrict__ dout, const int32_t *__restrict__ counters,
                                                 float *__restrict__ part) {
    constexpr int K = S == 3 ? kW2 : (S == 2 ? kW1 : kMaxK0);  // channels of block S's normalisation
    constexpr int NV = S == 1 ? 3 * 16 : 64;                    // staged columns with a per-channel sum
    constexpr int DH = 32, RR = S == 2 ? 64 : 48;               // staged dh and r (S = 2, 1)
    // pass 3 stages block 3's weight rows at a pitch of 36 floats (and a_2
    // after them): lanes that read different rows in the sparse loop then
    // fall on different LDS banks (at 32 they shared one)
    constexpr int kWP = 36, kA2P = S == 3 ? kW3 * kWP : kA2;
    __shared__ float Ps[kPadded];
    __shared__ float stg[64 * kStg];
    __shared__ int scl[64];
    extern __shared__ float tab[];  // per-cloud group sums, batched only: [kGnClouds][2 K] (launch size)
    const int lane = threadIdx.x;
    if (S == 3) {
        for (int i = lane; i < kW3 * kW2; i += 64) Ps[(i / kW2) * kWP + (i % kW2)] = P[kWt2 + i];
        for (int i = lane; i < kW2; i += 64) Ps[kA2P + i] = P[kA2 + i];
    } else {
        for (int i = lane; i < kPadded; i += 64) Ps[i] = P[i];
    }
    const bool tabbed = S != 1 && use_gn && BATCHED;
    if (tabbed)
        for (int i = lane; i < kGnClouds * 2 * K; i += 64) tab[i] = 0.f;
    // one cloud: its affines, normalisation and group means in LDS (the
    // lanes read them as broadcasts instead of a global load per channel)
    constexpr int kCst = kAffRow + kNrmRow + 2 * kW2 * 2;
    __shared__ float cst[BATCHED ? 1 : kCst];
    if (!BATCHED) {
        for (int i = lane; i < kAffRow; i += 64) cst[i] = aff[i];
        for (int i = lane; i < kNrmRow; i += 64) cst[kAffRow + i] = nrm[i];
        if (S != 3)  // the group means exist from pass 2 on
            for (int i = lane; i < 2 * kW2 * 2; i += 64) cst[kAffRow + kNrmRow + i] = gm[i];
    }
    __syncthreads();
    const int64_t E = counters[CNT_E];
    const int G = S == 3 ? G2 : G1;
    const int gs = K / G;                                       // channels per group (S = 3, 2)
    const int gs3 = kW2 / G2, gs2 = kW1 / G1;
    float vacc = 0.f;
    f32x16_t macc;
#pragma unroll
    for (int i = 0; i < 16; ++i) macc[i] = 0.f;
    float *st = stg + lane * kStg;
    for (int64_t e0 = (int64_t)blockIdx.x * 64; e0 < E; e0 += (int64_t)gridDim.x * 64) {
        const int64_t e = e0 + lane;
        const bool live = e < E;
        const int v = live ? lvert[e] : 0;
        const int cloud = BATCHED ? cloud_of(vkeys, 1, v) : 0;
        const float *A = BATCHED ? aff + (int64_t)cloud * kAffRow : cst;
        const float *N = BATCHED ? nrm + (int64_t)cloud * kNrmRow : cst + kAffRow;
        const float *GM = BATCHED ? gm + (int64_t)cloud * 2 * kW2 * 2 : cst + kAffRow + kNrmRow;
        const float *R = rec + (live ? e : 0) * kRec;
        // the part of the record this pass reads, as 16-byte loads (a lane's
        // record is 256 contiguous bytes)
        constexpr int RLO = S == 3 ? kRecH2 : (S == 2 ? kRecH1 : 0), RHI = S == 1 ? kRecH2 : kRec;
        float rv[kRec];
#pragma unroll
        for (int q = RLO / 4; q < RHI / 4; ++q) {
            const float4 t = reinterpret_cast<const float4 *>(R)[q];
            rv[4 * q] = t.x;
            rv[4 * q + 1] = t.y;
            rv[4 * q + 2] = t.z;
            rv[4 * q + 3] = t.w;
        }
        if (S == 3) {
            // dr3 = W3^T dh3, dh3 = g_v on the channels routed to this entry
            // (its mask) and 0 elsewhere: the row of g is loaded whole, and
            // the channels run in the same order in every lane, so that the
            // weights are LDS broadcasts
            const uint64_t mk = live ? routed[e] : 0ull;
            float gv[kW3];
            const float *grow = grad_out + (int64_t)v * kW3;
            if ((reinterpret_cast<uintptr_t>(grad_out) & 15) == 0) {  // 16-byte rows (uniform branch)
                const float4 *g4 = reinterpret_cast<const float4 *>(grow);
#pragma unroll
                for (int q = 0; q < kW3 / 4; ++q) {
                    const float4 t4 = g4[q];
                    gv[4 * q] = t4.x;
                    gv[4 * q + 1] = t4.y;
                    gv[4 * q + 2] = t4.z;
                    gv[4 * q + 3] = t4.w;
                }
            } else {
#pragma unroll
                for (int o = 0; o < kW3; ++o) gv[o] = grow[o];
            }
            float dr[kW2];
#pragma unroll
            for (int j = 0; j < kW2; ++j) dr[j] = 0.f;
            // Where every entry of the wavefront receives few channels (dense
            // vertices share their 64 channels among many entries), only the
            // set bits are visited, the row of g read back from this lane's
            // staging row; else all 64 channels, the weights as broadcasts.
            // The choice depends only on the data: repeated calls agree.
            int pc = __popcll(mk);
#pragma unroll
            for (int off = 32; off > 0; off >>= 1) pc = max(pc, __shfl_xor(pc, off));
            if (pc <= kSparseBits) {
#pragma unroll
                for (int o = 0; o < kW3; ++o) st[o] = gv[o];
                uint64_t bits = mk;
                while (bits) {
                    const int o = __builtin_ctzll(bits);
                    bits &= bits - 1;
                    const float g = st[o];
#pragma unroll
                    for (int j = 0; j < kW2; ++j) dr[j] = fmaf(g, Ps[o * kWP + j], dr[j]);
                }
            } else {
                // (fully unrolled: gv stays in registers)
#pragma unroll
                for (int o = 0; o < kW3; ++o) {
                    const float g = ((mk >> o) & 1ull) ? gv[o] : 0.f;
#pragma unroll
                    for (int j = 0; j < kW2; ++j) dr[j] = fmaf(g, Ps[o * kWP + j], dr[j]);
                }
            }
#pragma unroll
            for (int j = 0; j < kW2; ++j) {
                const float h = rv[kRecH2 + j];
                const float d = (live && fmaf(A[kAff2 + j], h, A[kAff2 + kW2 + j]) > 0.f) ? dr[j] : 0.f;
                const float xh = (h - N[2 * 64 + 2 * j]) * N[2 * 64 + 2 * j + 1];
                dr[j] = d;
                st[j] = d;
                st[kW2 + j] = d * xh;
            }
            if (live) {
                float4 *o4 = reinterpret_cast<float4 *>(dout + e * kW2);
#pragma unroll
                for (int q = 0; q < kW2 / 4; ++q) o4[q] = make_float4(dr[4 * q], dr[4 * q + 1], dr[4 * q + 2], dr[4 * q + 3]);
            }
        } else if (S == 2) {
            // block 3's input gradient dh2, then block 2: r2, dr2 = W2^T dh2, dhn2
            float dh[kW2];
            const float4 *i4 = reinterpret_cast<const float4 *>(din + (live ? e : 0) * kW2);
#pragma unroll
            for (int q = 0; q < kW2 / 4; ++q) {
                const float4 d4 = live ? i4[q] : make_float4(0.f, 0.f, 0.f, 0.f);
                dh[4 * q] = d4.x;
                dh[4 * q + 1] = d4.y;
                dh[4 * q + 2] = d4.z;
                dh[4 * q + 3] = d4.w;
            }
#pragma unroll
            for (int j = 0; j < kW2; ++j) {
                const float gj = Ps[kA2 + j] * dh[j];
                if (use_gn) {
                    const float xh = (rv[kRecH2 + j] - N[2 * 64 + 2 * j]) * N[2 * 64 + 2 * j + 1];
                    const float *M = GM + kW2 * 2 + (j / gs3) * 2;
                    dh[j] = live ? N[2 * 64 + 2 * j + 1] * (gj - M[0] - xh * M[1]) : 0.f;
                } else {
                    dh[j] = gj;
                }
                st[DH + j] = dh[j];
            }
            float dn[kW1];
#pragma unroll
            for (int c = 0; c < kW1; ++c) {
                const float h = rv[kRecH1 + c];
                const float hn = fmaf(A[kAff1 + c], h, A[kAff1 + kW1 + c]);
                float s_ = 0.f;
#pragma unroll
                for (int j = 0; j < kW2; ++j) s_ = fmaf(dh[j], Ps[kWt1 + j * kW1 + c], s_);
                const float d = hn > 0.f ? s_ : 0.f;
                const float xh = (h - N[1 * 64 + 2 * c]) * N[1 * 64 + 2 * c + 1];
                dn[c] = d;
                st[c] = d;
                st[kW1 + c] = d * xh;
                st[RR + c] = live ? relu(hn) : 0.f;
            }
            if (live) {
                float4 *o4 = reinterpret_cast<float4 *>(dout + e * kW1);
#pragma unroll
                for (int q = 0; q < kW1 / 4; ++q) o4[q] = make_float4(dn[4 * q], dn[4 * q + 1], dn[4 * q + 2], dn[4 * q + 3]);
            }
        } else {
            // block 2's input gradient dh1, then block 1: r1, dr1 = W1^T dh1, dhn1
            float dh[kW1];
            const float4 *i4 = reinterpret_cast<const float4 *>(din + (live ? e : 0) * kW1);
#pragma unroll
            for (int q = 0; q < kW1 / 4; ++q) {
                const float4 d4 = live ? i4[q] : make_float4(0.f, 0.f, 0.f, 0.f);
                dh[4 * q] = d4.x;
                dh[4 * q + 1] = d4.y;
                dh[4 * q + 2] = d4.z;
                dh[4 * q + 3] = d4.w;
            }
#pragma unroll
            for (int c = 0; c < kW1; ++c) {
                const float gc = Ps[kA1 + c] * dh[c];
                if (use_gn) {
                    const float xh = (rv[kRecH1 + c] - N[1 * 64 + 2 * c]) * N[1 * 64 + 2 * c + 1];
                    const float *M = GM + (c / gs2) * 2;
                    dh[c] = live ? N[1 * 64 + 2 * c + 1] * (gc - M[0] - xh * M[1]) : 0.f;
                } else {
                    dh[c] = gc;
                }
                st[DH + c] = dh[c];
            }
#pragma unroll
            for (int c = 0; c < kMaxK0; ++c) {
                const float h = rv[c];
                const float hn = fmaf(A[kAff0 + c], h, A[kAff0 + kMaxK0 + c]);
                float s_ = 0.f;
#pragma unroll
                for (int o = 0; o < kW1; ++o) s_ = fmaf(dh[o], Ps[kWt0 + o * kMaxK0 + c], s_);
                const float d = hn > 0.f ? s_ : 0.f;
                st[c] = d;
                st[kMaxK0 + c] = d * ((h - N[2 * c]) * N[2 * c + 1]);
                st[RR + c] = live ? relu(hn) : 0.f;
            }
        }
        scl[lane] = live ? cloud : -1;
        __syncthreads();
        // per-channel sums: lane c adds column c, entries in order
        if (lane < NV) {
#pragma unroll 8
            for (int k = 0; k < 64; ++k) vacc += stg[k * kStg + lane];
        }
        // batched group sums: lane (group, part) adds each entry to its cloud
        if (tabbed && lane < 2 * G) {
            const int grp = lane >> 1, pt = lane & 1;
            for (int k = 0; k < 64; ++k) {
                const int cl = scl[k];
                if (cl < 0) continue;
                float x = 0.f;
                for (int t = 0; t < gs; ++t) {
                    const int ch = grp * gs + t;
                    x = fmaf(Ps[(S == 3 ? kA2P : kA1) + ch], stg[k * kStg + pt * K + ch], x);
                }
                tab[cl * 2 * K + lane] += x;
            }
        }
        // weight gradient: two entries a step, dh rows as A, r rows as B
        if (S != 3) {
            const int i = lane & 31, half = lane >> 5;
#pragma unroll 4
            for (int s2 = 0; s2 < 32; ++s2) {
                const float *row = stg + (2 * s2 + half) * kStg;
                const float a = (S == 2 || i < kW1) ? row[DH + (i & (S == 2 ? 31 : 15))] : 0.f;
                const float b = i < 16 ? row[RR + (i & 15)] : 0.f;
                macc = __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, macc, 0, 0, 0);
            }
        }
        __syncthreads();  // the staging is rewritten by the next chunk
    }

    // the wavefront's partial row
    const int np = pb_len(S, batched);
    float *out = part + (int64_t)blockIdx.x * np;
    if (S == 3) {
        out[lane < kW2 ? kW2 + lane : lane - kW2] = vacc;  // dbeta3 (columns 0..31), dgamma3 (32..63)
    } else if (S == 2) {
        if (lane < kW1) out[kW2 * kW1 + kW2 + kW1 + lane] = vacc;                  // dbeta2
        else if (lane < 2 * kW1) out[kW2 * kW1 + kW2 + (lane - kW1)] = vacc;       // dgamma2
        else out[kW2 * kW1 + (lane - 2 * kW1)] = vacc;                             // db2
    } else {
        if (lane < kMaxK0) out[kW1 * kMaxK0 + kW1 + kMaxK0 + lane] = vacc;         // dbeta1
        else if (lane < 2 * kMaxK0) out[kW1 * kMaxK0 + kW1 + (lane - kMaxK0)] = vacc;  // dgamma1
        else if (lane < 3 * kMaxK0) out[kW1 * kMaxK0 + (lane - 2 * kMaxK0)] = vacc;    // db1
    }
    if (S != 3) {
        // the MFMA tile: lane l holds column l mod 32, register r row
        // 8 (r / 4) + 4 (l / 32) + r mod 4
        const int j = lane & 31;
        constexpr int NI = S == 2 ? kW2 : kW1, NJ = S == 2 ? kW1 : kMaxK0;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int i = 8 * (r / 4) + 4 * (lane >> 5) + (r & 3);
            if (i < NI && j < NJ) out[i * NJ + j] = macc[r];
        }
    }
    if (S != 1 && use_gn) {
        const int base = S == 3 ? kPB3Base : kPB2Base;
        if (tabbed) {
            __syncthreads();
            for (int i = lane; i < kGnClouds * 2 * K; i += 64) out[base + i] = tab[i];
        } else {
            // one cloud: group sum = sum over the group's channels of gamma
            // times the per-channel sum (dbeta's column, or dgamma's: dbeta
            // in lane ch, dgamma in lane K + ch)
            const int grp = lane >> 1, pt = lane & 1;
            float x = 0.f;
            for (int t = 0; t < gs; ++t) {
                const int ch = (grp < G ? grp : 0) * gs + t;
                const float y = __shfl(vacc, pt * K + ch);
                x = fmaf(Ps[(S == 3 ? kA2P : kA1) + ch], y, x);
            }
            if (lane < 2 * K) out[base + lane] = grp < G ? x : 0.f;
        }
    } else if (S != 1) {
        const int base = S == 3 ? kPB3Base : kPB2Base;
        for (int i = lane; i < np - base; i += 64) out[base + i] = 0.f;
    }
}

// The group means of block l's (l = 1: block 2, l = 2: block 3) gradient
// sums: gm[cloud][l - 1][group] = (sum gn, sum gn xhat) / (rows * group size).
__global__ __launch_bounds__(kBlock) void k_dpn_gnmean(const float *__restrict__ sums, int l, int G,
                                                       const double *__restrict__ rows,
                                                       const int32_t *__restrict__ counters, int batched,
                                                       float *__restrict__ gm) {
    const int K = l == 2 ? kW2 : kW1;
    const int gsz = K / G;
    const int nc = num_clouds(counters, batched);  // the clouds k_dpn_norm counted
    for (int i = threadIdx.x + blockIdx.x * kBlock; i < nc * G; i += gridDim.x * kBlock) {
        const int b = i / G, gi = i % G;
        const double n = rows[b] * gsz;
        const float *s = sums + (b * K + gi) * 2;
        float *o = gm + ((int64_t)b * 2 + (l - 1)) * kW2 * 2 + gi * 2;
        o[0] = n > 0.0 ? (float)(s[0] / n) : 0.f;
        o[1] = n > 0.0 ? (float)(s[1] / n) : 0.f;
    }
}

// The reduced sums in the caller's layout: per block, d(gamma or a) [K],
// d(beta or s) [K], dW [w][K], db [w].
__global__ __launch_bounds__(kBlock) void k_dpn_out(const float *__restrict__ r1, const float *__restrict__ r2,
                                                    const float *__restrict__ r3, const float *__restrict__ rarg,
                                                    int k0, float *__restrict__ grad) {
    const int n1 = 2 * k0 + kW1 * k0 + kW1, n2 = 2 * kW1 + kW2 * kW1 + kW2, n3 = 2 * kW2 + kW3 * kW2 + kW3;
    for (int i = threadIdx.x + blockIdx.x * kBlock; i < n1 + n2 + n3; i += gridDim.x * kBlock) {
        float x;
        if (i < n1) {
            if (i < k0) x = r1[kW1 * kMaxK0 + kW1 + i];
            else if (i < 2 * k0) x = r1[kW1 * kMaxK0 + kW1 + kMaxK0 + (i - k0)];
            else if (i < 2 * k0 + kW1 * k0) {
                const int o = (i - 2 * k0) / k0, c = (i - 2 * k0) % k0;
                x = r1[o * kMaxK0 + c];
            } else {
                x = r1[kW1 * kMaxK0 + (i - 2 * k0 - kW1 * k0)];
            }
        } else if (i < n1 + n2) {
            const int j = i - n1;
            if (j < 2 * kW1) x = r2[kW2 * kW1 + kW2 + j];          // dgamma2, dbeta2
            else if (j < 2 * kW1 + kW2 * kW1) x = r2[j - 2 * kW1];  // dW2
            else x = r2[kW2 * kW1 + (j - 2 * kW1 - kW2 * kW1)];     // db2
        } else {
            const int j = i - n1 - n2;
            if (j < 2 * kW2) x = r3[j];                              // dgamma3, dbeta3
            else if (j < 2 * kW2 + kW3 * kW2) x = rarg[j - 2 * kW2]; // dW3
            else x = rarg[kW3 * kW2 + (j - 2 * kW2 - kW3 * kW2)];    // db3
        }
        grad[i] = x;
    }
}

}  // namespace

// Packed parameter count for d + f_d = k0 inputs: per block a [K], s [K],
// W [w][K], b [w] with K the block's input width.
int pointnet_padded_count() { return kPadded; }

int pointnet_param_count(int k0) {
    return 2 * k0 + kW1 * k0 + kW1 + 2 * kW1 + kW2 * kW1 + kW2 + 2 * kW2 + kW3 * kW2 + kW3;
}

// Bytes of the statistics (every copy of every cloud's row) and of the
// affines (one row per cloud).
int64_t pointnet_stats_bytes() { return (int64_t)kStatRows * kStatRow * (int64_t)sizeof(double); }
int64_t pointnet_aff_bytes() { return (int64_t)kGnClouds * kAffRow * (int64_t)sizeof(float); }

hipError_t launch_distribute_pointnet(lattice *L, const float *pos, const float *feat, int f_d, const float *params,
                                      const int *groups, float eps, void *out, bool out_bf16, float *mean) {
    if (L->m == 0) return hipSuccess;
    const int d = L->d;
    const int k0 = d + f_d;
    const int batched = (groups && L->batched) ? 1 : 0;  // per-cloud statistics
    float *mu = mean ? mean : L->mu;
    const int64_t E = L->m * (int64_t)(d + 1);
    const unsigned g_v = grid_for(L->max_vertices, kBlock, L->cu_count, 8);
    hipLaunchKernelGGL(k_entry_vertex, dim3(g_v), dim3(kBlock), 0, L->stream, L->vinfo, L->split, L->rowmap,
                       L->vkeys, batched, L->counters, d, L->lvert, L->macc);
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
    const unsigned g_z = groups ? grid_for((int64_t)kStatRows * kStatRow, kBlock, L->cu_count, 1) : 1;
    hipLaunchKernelGGL(k_pointnet_prep, dim3(g_v + g_i + g_k + g_z), dim3(kBlock), 0, L->stream, L->vinfo, L->macc,
                       d, L->counters, mu, L->lvert, L->pn_keys, params, k0, L->pn_params, groups ? 1 : 0, batched,
                       L->pn_stats, L->pn_aff, (int)g_v, (int)g_i, (int)g_k, (int)g_z);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    const unsigned g_p = grid_for(E, kBlock, L->cu_count, 2);  // 69 KB of LDS: two workgroups per CU
    if (groups) {
        const int widths[3] = {k0, kW1, kW2};
        auto finalize = [&](int l) {
            const int kp = l == 2 ? kW2 : kMaxK0;
            const unsigned g_f = grid_for((int64_t)(batched ? kGnClouds : 1) * kp * 64, kBlock, L->cu_count, 1);
            hipLaunchKernelGGL(k_gn_finalize, dim3(g_f), dim3(kBlock), 0, L->stream, L->pn_stats, L->pn_params,
                               L->counters, batched, l, widths[l], groups[l], eps, L->pn_aff);
            return hipGetLastError();
        };
        // two workgroups per CU: each wavefront's range of chunks is long
        // enough that its one hand-over of the sums is a small part of it
        const unsigned g_s = grid_for(E, kBlock, L->cu_count, 2);
        switch (d) {
#define GS_CASE(DD)                                                                                                \
    case DD:                                                                                                       \
        hipLaunchKernelGGL(k_gn_stats0<DD>, dim3(g_s), dim3(kBlock), 0, L->stream, L->list, L->lvert, L->vkeys,    \
                           batched, pos, feat, f_d, mu, L->counters, L->pn_stats);                                 \
        break;
            GS_CASE(1)
            GS_CASE(2)
            GS_CASE(3)
            GS_CASE(4)
#undef GS_CASE
            default:
                return hipErrorInvalidValue;
        }
        if ((e = hipGetLastError()) != hipSuccess) return e;
        if ((e = finalize(0)) != hipSuccess) return e;
        hipLaunchKernelGGL((k_pointnet<1, false>), dim3(g_p), dim3(kBlock), 0, L->stream, L->list, L->lvert, L->vinfo,
                           L->vkeys, batched, pos, feat, d, f_d, L->pn_params, L->pn_aff, mu, L->counters,
                           L->pn_stats, L->pn_keys, out, nullptr, nullptr, nullptr, nullptr);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        if ((e = finalize(1)) != hipSuccess) return e;
        hipLaunchKernelGGL((k_pointnet<2, false>), dim3(g_p), dim3(kBlock), 0, L->stream, L->list, L->lvert, L->vinfo,
                           L->vkeys, batched, pos, feat, d, f_d, L->pn_params, L->pn_aff, mu, L->counters,
                           L->pn_stats, L->pn_keys, out, nullptr, nullptr, nullptr, nullptr);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        if ((e = finalize(2)) != hipSuccess) return e;
    }
    hipLaunchKernelGGL((out_bf16 ? k_pointnet<3, true> : k_pointnet<3, false>), dim3(g_p), dim3(kBlock), 0, L->stream,
                       L->list, L->lvert, L->vinfo, L->vkeys, batched, pos, feat, d, f_d, L->pn_params, L->pn_aff, mu,
                       L->counters, L->pn_stats, L->pn_keys, out, nullptr, nullptr, nullptr, nullptr);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL((out_bf16 ? k_pointnet_rows<true> : k_pointnet_rows<false>), dim3(g_i), dim3(kBlock), 0,
                       L->stream, L->lvert, L->vinfo, L->counters, L->pn_keys, out);
    return hipGetLastError();
}

// Scratch of the backward (offsets in bytes, 256-aligned).
struct DpnLayout {
    int64_t out, rec, routed, win, wslot, d3, d2, nrm, rows, gm, parg, pb3, pb2, pb1, r3, r2, r1, rarg, tmp, total;
    int nwaves_arg, nwaves;
};

static DpnLayout dpn_layout(const lattice *L) {
    auto al = [](int64_t x) { return (x + 255) / 256 * 256; };
    DpnLayout l;
    l.nwaves_arg = L->cu_count * 4 * kWaves;  // four workgroups of four wavefronts per CU
    l.nwaves = L->cu_count * 4;               // backward passes: four one-wavefront workgroups per CU
    const int64_t V = L->max_vertices, E = (int64_t)(L->d + 1) * L->max_points;
    int64_t at = 0;
    l.out = at;    at += al(V * kW3 * 4);
    l.rec = at;    at += al(E * kRec * 4);
    l.routed = at; at += al(E * 8);
    l.win = at;    at += al(V * kW3 * 4);
    l.wslot = at;  at += al((E + 63) / 64 * 2 * kW3 * 8);
    l.d3 = at;     at += al(E * kW2 * 4);
    l.d2 = at;     at += al(E * kW1 * 4);
    l.nrm = at;    at += al((int64_t)kGnClouds * kNrmRow * 4);
    l.rows = at;   at += al((int64_t)kGnClouds * 8);
    l.gm = at;     at += al((int64_t)kGnClouds * 2 * kW2 * 2 * 4);
    l.parg = at;   at += al((int64_t)l.nwaves_arg * kPArg * 4);
    l.pb3 = at;    at += al((int64_t)l.nwaves * kPB3 * 4);
    l.pb2 = at;    at += al((int64_t)l.nwaves * kPB2 * 4);
    l.pb1 = at;    at += al((int64_t)l.nwaves * kPB1 * 4);
    l.r3 = at;     at += al(kPB3 * 4);
    l.r2 = at;     at += al(kPB2 * 4);
    l.r1 = at;     at += al(kPB1 * 4);
    l.rarg = at;   at += al(kPArg * 4);
    int64_t t = rowsum::scratch_floats(l.nwaves_arg, kPArg);
    for (int64_t n : {kPB3, kPB2, kPB1})
        if (rowsum::scratch_floats(l.nwaves, n) > t) t = rowsum::scratch_floats(l.nwaves, n);
    l.tmp = at;    at += al(t * 4);
    l.total = at;
    return l;
}

int64_t pointnet_backward_scratch_bytes(const lattice *L) { return dpn_layout(L).total; }

hipError_t launch_distribute_backward(lattice *L, const float *pos, const float *feat, int f_d, const float *params,
                                      const int *groups, float eps, const float *grad_out, float *grad_params,
                                      void *scratch) {
    if (L->m == 0)  // no rows: every gradient is zero (a sum of no rows)
        return rowsum::sum(L->stream, grad_params, 0, pointnet_param_count(L->d + f_d), nullptr, grad_params);
    const DpnLayout l = dpn_layout(L);
    char *s = reinterpret_cast<char *>(scratch);
    auto F = [&](int64_t off) { return reinterpret_cast<float *>(s + off); };
    const int k0 = L->d + f_d;
    const int use_gn = groups ? 1 : 0;
    const int batched = (groups && L->batched) ? 1 : 0;
    const int G0 = groups ? groups[0] : 1, G1 = groups ? groups[1] : 1, G2 = groups ? groups[2] : 1;
    // the forward: entry-to-vertex map, local means, statistics and affines
    hipError_t e = launch_distribute_pointnet(L, pos, feat, f_d, params, groups, eps, F(l.out), false, nullptr);
    if (e != hipSuccess) return e;
    double *rows = reinterpret_cast<double *>(s + l.rows);
    hipLaunchKernelGGL(k_dpn_norm, dim3((unsigned)((kGnClouds * 96 + kWaves - 1) / kWaves)), dim3(kBlock), 0,
                       L->stream, L->pn_stats, L->counters, batched, use_gn, k0, G0, G1, G2, eps, F(l.nrm), rows);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    // the per-entry records (h_0 .. h_3) by the forward's own MFMA pass, so
    // that the argmax sees exactly the values the forward's max took
    uint64_t *routed = reinterpret_cast<uint64_t *>(s + l.routed);
    const unsigned g_p = grid_for((int64_t)(L->d + 1) * L->m, kBlock, L->cu_count, 2);
    hipLaunchKernelGGL((k_pointnet<4, false>), dim3(g_p), dim3(kBlock), 0, L->stream, L->list, L->lvert, L->vinfo,
                       L->vkeys, batched, pos, feat, L->d, f_d, L->pn_params, L->pn_aff, L->mu, L->counters,
                       L->pn_stats, L->pn_keys, nullptr, F(l.rec), routed, reinterpret_cast<int32_t *>(s + l.win),
                       reinterpret_cast<uint2 *>(s + l.wslot));
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(k_dpn_argmax, dim3((unsigned)(l.nwaves_arg / kWaves)), dim3(kBlock), 0, L->stream, L->vinfo,
                       L->vkeys, batched, L->pn_aff, F(l.rec), reinterpret_cast<const int32_t *>(s + l.win),
                       reinterpret_cast<const uint2 *>(s + l.wslot), grad_out, L->counters, routed, F(l.parg));
    if ((e = hipGetLastError()) != hipSuccess) return e;
    auto reduce = [&](const float *part, int64_t nrows, int64_t n, float *out) {
        return rowsum::sum(L->stream, part, nrows, n, F(l.tmp), out);
    };
    auto back = [&](auto kern, int K, const float *din, float *dout, int64_t part_off) {
        const size_t tab = (use_gn && batched && K > 0) ? (size_t)kGnClouds * 2 * K * sizeof(float) : 0;
        hipLaunchKernelGGL(kern, dim3((unsigned)l.nwaves), dim3(64), tab, L->stream, L->lvert, L->vkeys, batched,
                           use_gn, G1, G2, L->pn_params, L->pn_aff, F(l.nrm), F(l.gm), F(l.rec), routed, grad_out,
                           din, dout, L->counters, F(part_off));
        return hipGetLastError();
    };
    auto gnmean = [&](const float *sums, int lb, int G) {
        hipLaunchKernelGGL(k_dpn_gnmean, dim3(1), dim3(kBlock), 0, L->stream, sums, lb, G, rows, L->counters, batched,
                           F(l.gm));
        return hipGetLastError();
    };
    if ((e = batched ? back(k_dpn_back<3, true>, kW2, nullptr, F(l.d3), l.pb3)
                   : back(k_dpn_back<3, false>, kW2, nullptr, F(l.d3), l.pb3)) != hipSuccess)
        return e;
    if ((e = reduce(F(l.pb3), l.nwaves, pb_len(3, batched), F(l.r3))) != hipSuccess) return e;
    if (use_gn && (e = gnmean(F(l.r3) + kPB3Base, 2, G2)) != hipSuccess) return e;
    if ((e = batched ? back(k_dpn_back<2, true>, kW1, F(l.d3), F(l.d2), l.pb2)
                   : back(k_dpn_back<2, false>, kW1, F(l.d3), F(l.d2), l.pb2)) != hipSuccess)
        return e;
    if ((e = reduce(F(l.pb2), l.nwaves, pb_len(2, batched), F(l.r2))) != hipSuccess) return e;
    if (use_gn && (e = gnmean(F(l.r2) + kPB2Base, 1, G1)) != hipSuccess) return e;
    if ((e = batched ? back(k_dpn_back<1, true>, 0, F(l.d2), nullptr, l.pb1)
                   : back(k_dpn_back<1, false>, 0, F(l.d2), nullptr, l.pb1)) != hipSuccess)
        return e;
    if ((e = reduce(F(l.pb1), l.nwaves, kPB1, F(l.r1))) != hipSuccess) return e;
    if ((e = reduce(F(l.parg), l.nwaves_arg, kPArg, F(l.rarg))) != hipSuccess) return e;
    hipLaunchKernelGGL(k_dpn_out, dim3(16), dim3(kBlock), 0, L->stream, F(l.r1), F(l.r2), F(l.r3), F(l.rarg), k0,
                       grad_params);
    return hipGetLastError();
}
