// 1-hop-ring lattice convolution (Sec. "Common Operations on Permutohedral
// Lattice", Convolving; an unallocated neighbour contributes zero):
//   y_v[o] = bias[o] + sum_t sum_i x_{nbr(v,t)}[i] W[o][t][i].
//
// After the gather this is one dense product Y[V x C_out] = Z[V x K] W^T with
// K = T C_in, where row v of Z is the concatenation of the T neighbour rows.
// Both Z (gathered rows) and W ([C_out][T][C_in]) are K-contiguous, which is
// the operand layout the MFMA instructions consume.
//
// k_conv_mfma: a workgroup owns a BM x BN output tile and walks K in chunks
// of 128 LDS bytes per row (64 bf16 or 32 fp32 channels of one tap).  Per
// chunk it gathers the BM neighbour rows and the BN weight rows from global
// memory into registers, stages them in LDS (two buffers), and each wavefront
// computes a WR x WC sub-tile as MFMA 32x32 blocks.  The register stage is a
// ring of P chunks: the loads of chunk q+P are issued before chunk q is
// multiplied, so P chunks of gathers are in flight while the matrix cores
// work.  Three input modes:
//   CM 0  fp32 rows, fp32 MFMA (32x32x2)
//   CM 1  fp32 rows rounded to bf16 while staging, bf16 MFMA (32x32x16)
//   CM 2  bf16 rows (already rounded by their producer), bf16 MFMA
// The output is fp32 or, rounded to nearest even, bf16.  The tile loop is
// persistent: V lives on the device, so the grid is sized for the largest
// lattice and every workgroup reads V and strides over the tiles.
//
// k_conv_generic: one thread per output element, for channel counts the MFMA
// tiling does not cover (e.g. 8 -> 16).
#include "internal.h"

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

// fp32 -> bf16 bits, round to nearest with ties to even (NaN stays a quiet NaN).
__device__ __forceinline__ uint32_t bf16_bits(float f) {
    const uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (u >> 16) | 0x40u;
    return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}

__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

constexpr int kRowBytes = 144;  // one LDS row: 128 bytes of K plus 16 bytes of padding

// Largest tap count (d = 4): the tile's neighbour rows are staged in LDS.
constexpr int kMaxTaps = LATTICE_TAPS(LATTICE_MAX_D);

template <int CM, bool OUT_BF16, int BM, int BN, int WR, int WC, int P>
__global__ __launch_bounds__((BM / WR) * (BN / WC) * 64) void k_conv_mfma(
    const void *__restrict__ in, int C_in, const void *__restrict__ wv, int C_out, int T,
    const float *__restrict__ bias, void *__restrict__ out, const int32_t *__restrict__ nbr,
    const int32_t *__restrict__ counters) {
    constexpr bool BF16 = CM != 0;
    constexpr int WN = BN / WC;                   // wavefronts along N
    constexpr int NT = (BM / WR) * WN * 64;
    constexpr int TI = WR / 32;                   // MFMA blocks per wave along M
    constexpr int TJ = WC / 32;                   // MFMA blocks per wave along N
    constexpr int KC = BF16 ? 64 : 32;            // K elements per chunk (128 bytes of LDS row)
    constexpr int IN_ESZ = CM == 2 ? 2 : 4;       // bytes per stored input element
    constexpr int A_SEGS = KC * IN_ESZ / 16;      // 16-byte source segments per gathered row
    constexpr int A_RPP = NT / A_SEGS;            // gathered rows per pass
    constexpr int A_PASSES = BM / A_RPP;
    constexpr int B_RPP = NT / 8;                 // weight rows per pass (8 x 16 B per row)
    constexpr int B_PASSES = BN / B_RPP;
    constexpr int W_ESZ = BF16 ? 2 : 4;
    static_assert(A_PASSES * A_RPP == BM, "A tiling");
    static_assert(B_PASSES * B_RPP == BN, "B tiling");

    __shared__ __attribute__((aligned(16))) char lds[2 * (BM + BN) * kRowBytes];
    __shared__ int32_t nbr_s[BM * kMaxTaps];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave / WN;
    const int wn = wave % WN;
    const int64_t V = counters[CNT_V];
    const int64_t n_mt = (V + BM - 1) / BM;
    const int n_nt = C_out / BN;
    const int64_t ntiles = n_mt * n_nt;
    const int64_t K = (int64_t)T * C_in;
    const int CPT = C_in / KC;
    const int NQ = T * CPT;

    const int a_seg = tid % A_SEGS;
    const int a_row0 = tid / A_SEGS;
    const int b_seg = tid & 7;
    const int b_row0 = tid >> 3;
    const int lrow = lane & 31;
    const int khalf = lane >> 5;

    for (int64_t tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
        const int64_t row_base = (tile / n_nt) * BM;
        const int col_base = (int)(tile % n_nt) * BN;

        // The tile's neighbour rows are one contiguous run of BM * T indices.
        for (int i = tid; i < BM * T; i += NT) {
            const int64_t e = row_base * T + i;
            nbr_s[i] = (e < V * T) ? nbr[e] : -1;
        }
        __syncthreads();

        f32x16_t acc[TI][TJ];
#pragma unroll
        for (int i = 0; i < TI; ++i)
#pragma unroll
            for (int j = 0; j < TJ; ++j)
#pragma unroll
                for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

        u32x4_t areg[P][A_PASSES];
        u32x4_t breg[P][B_PASSES];
        bool present[P][A_PASSES];

        // Branch-free gather into ring slot s: an absent neighbour reads row 0
        // (V >= 1 whenever a tile exists) and is zeroed when it is written to
        // LDS, so the loads stay in flight until then.
        auto load_chunk = [&](int q, int s) {
            const int t = q / CPT;
            const int c0 = (q - t * CPT) * KC;
#pragma unroll
            for (int i = 0; i < A_PASSES; ++i) {
                const int u = nbr_s[(a_row0 + i * A_RPP) * T + t];
                present[s][i] = u >= 0;
                const int64_t row = u >= 0 ? u : 0;
                areg[s][i] = *reinterpret_cast<const u32x4_t *>(reinterpret_cast<const char *>(in) +
                                                                (row * C_in + c0) * IN_ESZ + a_seg * 16);
            }
#pragma unroll
            for (int i = 0; i < B_PASSES; ++i) {
                const int64_t n = col_base + b_row0 + i * B_RPP;
                breg[s][i] = *reinterpret_cast<const u32x4_t *>(reinterpret_cast<const char *>(wv) +
                                                                (n * K + (int64_t)t * C_in + c0) * W_ESZ + b_seg * 16);
            }
        };
        auto store_chunk = [&](int s, int buf) {
            char *A = lds + buf * (BM + BN) * kRowBytes;
            char *B = A + BM * kRowBytes;
#pragma unroll
            for (int i = 0; i < A_PASSES; ++i) {
                const int row = a_row0 + i * A_RPP;
                const u32x4_t x = present[s][i] ? areg[s][i] : u32x4_t{0u, 0u, 0u, 0u};
                if (CM == 1) {
                    u32x2_t pk;
                    pk[0] = bf16_bits(__uint_as_float(x[0])) | (bf16_bits(__uint_as_float(x[1])) << 16);
                    pk[1] = bf16_bits(__uint_as_float(x[2])) | (bf16_bits(__uint_as_float(x[3])) << 16);
                    *reinterpret_cast<u32x2_t *>(A + row * kRowBytes + a_seg * 8) = pk;
                } else {
                    *reinterpret_cast<u32x4_t *>(A + row * kRowBytes + a_seg * 16) = x;
                }
            }
#pragma unroll
            for (int i = 0; i < B_PASSES; ++i) {
                const int n = b_row0 + i * B_RPP;
                *reinterpret_cast<u32x4_t *>(B + n * kRowBytes + b_seg * 16) = breg[s][i];
            }
        };
        auto compute = [&](int buf) {
            const char *A = lds + buf * (BM + BN) * kRowBytes;
            const char *B = A + BM * kRowBytes;
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int boff = g * 32 + khalf * 16;
                u32x4_t a[TI], b[TJ];
#pragma unroll
                for (int i = 0; i < TI; ++i)
                    a[i] = *reinterpret_cast<const u32x4_t *>(A + (wm * WR + i * 32 + lrow) * kRowBytes + boff);
#pragma unroll
                for (int j = 0; j < TJ; ++j)
                    b[j] = *reinterpret_cast<const u32x4_t *>(B + (wn * WC + j * 32 + lrow) * kRowBytes + boff);
                if (BF16) {
#pragma unroll
                    for (int i = 0; i < TI; ++i)
#pragma unroll
                        for (int j = 0; j < TJ; ++j)
                            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                                __builtin_bit_cast(bf16x8_t, a[i]), __builtin_bit_cast(bf16x8_t, b[j]), acc[i][j], 0,
                                0, 0);
                } else {
                    // Lane half h holds k = g*8 + 4h + c in component c; step c
                    // pairs the same components of A and B, so every k meets its
                    // own weight exactly once.
#pragma unroll
                    for (int c = 0; c < 4; ++c)
#pragma unroll
                        for (int i = 0; i < TI; ++i)
#pragma unroll
                            for (int j = 0; j < TJ; ++j)
                                acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(
                                    __uint_as_float(a[i][c]), __uint_as_float(b[j][c]), acc[i][j], 0, 0, 0);
                }
            }
        };

        // Prologue: chunks 0..P-1 into the ring, chunk 0 into LDS buffer 0.
#pragma unroll
        for (int s = 0; s < P; ++s)
            if (s < NQ) load_chunk(s, s);
        store_chunk(0, 0);
        __syncthreads();
        // Steady state, free of branches so that the compiler keeps the ring's
        // loads in flight across iterations: past the last chunk the refill
        // re-reads chunk NQ-1 and the store writes an LDS buffer nobody reads.
        const int NQP = (NQ / P) * P;
        for (int q0 = 0; q0 < NQP; q0 += P) {
#pragma unroll
            for (int s = 0; s < P; ++s) {
                const int q = q0 + s;
                // ring slot s held chunk q, already in LDS: refill it with chunk q+P
                load_chunk(q + P < NQ ? q + P : NQ - 1, s);
                compute(q & 1);
                store_chunk((s + 1) % P, (q + 1) & 1);
                __syncthreads();
            }
        }
        // Remainder (fewer than P chunks, all already loaded).
#pragma unroll
        for (int s = 0; s < P; ++s) {
            const int q = NQP + s;
            if (q < NQ) {
                compute(q & 1);
                if (q + 1 < NQ) store_chunk((s + 1) % P, (q + 1) & 1);
                __syncthreads();
            }
        }

        // 32x32 accumulator layout: register r of lane l holds
        // row 8 (r / 4) + 4 (l / 32) + r % 4, column l % 32.
#pragma unroll
        for (int i = 0; i < TI; ++i)
#pragma unroll
            for (int j = 0; j < TJ; ++j) {
                const int col = col_base + wn * WC + j * 32 + lrow;
                const float bc = bias ? bias[col] : 0.f;
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int64_t row = row_base + wm * WR + i * 32 + 8 * (r >> 2) + 4 * khalf + (r & 3);
                    if (row < V) {
                        const float y = acc[i][j][r] + bc;
                        if (OUT_BF16)
                            reinterpret_cast<uint16_t *>(out)[row * C_out + col] = (uint16_t)bf16_bits(y);
                        else
                            reinterpret_cast<float *>(out)[row * C_out + col] = y;
                    }
                }
            }
    }
}

// Weight-stationary variant: the workgroup's slice of W (BN output channels,
// all K = T C_in) stays in LDS for the whole persistent loop, and every
// wavefront independently computes 32-row x BN tiles, gathering its A rows
// straight into MFMA operand registers (16 bytes per lane per k-group) PT taps
// ahead of their use.  No barrier in the main loop.  The tap loop is unrolled
// (T is a template parameter).  CM as for k_conv_mfma.  For the fp32 MFMA
// (32x32x2), lane half h holds k = 8 g + 4 h + c in component c of its A and
// B registers; step c pairs the same components, so every k meets its own
// weight exactly once.
template <int CM, bool OUT_BF16, int T, int C_IN, int CB, int PT>
__global__ __launch_bounds__(512) void k_conv_ws(const void *__restrict__ in, const void *__restrict__ wv, int C_out,
                                                 const float *__restrict__ bias, void *__restrict__ out,
                                                 const int32_t *__restrict__ nbr, const int32_t *__restrict__ counters) {
    constexpr bool BF16 = CM != 0;
    constexpr int NW = 8;                        // wavefronts per workgroup
    constexpr int BN = 32 * CB;
    constexpr int K = T * C_IN;
    constexpr int WESZ = BF16 ? 2 : 4;
    constexpr int KSTRIDE = K * WESZ + 16;       // LDS bytes per weight row (16 B pad: no bank conflicts)
    constexpr int KGE = BF16 ? 16 : 8;           // K elements per k-group
    constexpr int KG = C_IN / KGE;               // k-groups per tap
    constexpr int IN_ESZ = CM == 2 ? 2 : 4;
    constexpr int AW = CM == 1 ? 2 : 1;          // 16-byte loads per lane per k-group (fp32 rows -> bf16)
    static_assert(C_IN % KGE == 0, "channels");
    extern __shared__ __attribute__((aligned(16))) char wlds[];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int lrow = lane & 31;
    const int khalf = lane >> 5;
    const int n_nt = C_out / BN;
    const int nt = blockIdx.x % n_nt;
    const int col_base = nt * BN;
    const int64_t V = counters[CNT_V];
    const int64_t n_mt = (V + 31) / 32;

    // W slice -> LDS, once: every load of the slice is issued before the
    // first store so that their latencies overlap (a load-store loop would
    // wait out one latency per 8 KB).  The first tile's neighbour indices
    // are fetched in the same window.
    const int64_t wave0 = (int64_t)(blockIdx.x / n_nt) * NW + wave;
    const int64_t nwaves = (int64_t)(gridDim.x / n_nt) * NW;
    int nbn[T];
    {
        const int64_t row = wave0 * 32 + lrow;
        const bool live = row < V;
#pragma unroll
        for (int t = 0; t < T; ++t) nbn[t] = live ? nbr[row * T + t] : -1;
    }
    {
        constexpr int SEGS = K * WESZ / 16;
        constexpr int TOTAL = BN * SEGS;
        constexpr int PER = (TOTAL + NW * 64 - 1) / (NW * 64);
        const char *src = reinterpret_cast<const char *>(wv) + (int64_t)col_base * K * WESZ;
        u32x4_t wr[PER];
#pragma unroll
        for (int q = 0; q < PER; ++q) {
            const int i = tid + q * NW * 64;
            if (i < TOTAL) {
                const int n = i / SEGS, sg = i - n * SEGS;
                wr[q] = *reinterpret_cast<const u32x4_t *>(src + (int64_t)n * K * WESZ + sg * 16);
            }
        }
#pragma unroll
        for (int q = 0; q < PER; ++q) {
            const int i = tid + q * NW * 64;
            if (i < TOTAL) {
                const int n = i / SEGS, sg = i - n * SEGS;
                *reinterpret_cast<u32x4_t *>(wlds + n * KSTRIDE + sg * 16) = wr[q];
            }
        }
    }
    __syncthreads();

    for (int64_t mt = wave0; mt < n_mt; mt += nwaves) {
        // With up to two accumulator blocks, this tile's neighbour indices
        // were fetched before it and the next tile's are fetched now; four
        // blocks leave too few registers for that.
        int nb[T];
        if constexpr (CB < 4) {
#pragma unroll
            for (int t = 0; t < T; ++t) nb[t] = nbn[t];
            const int64_t row = (mt + nwaves) * 32 + lrow;
            const bool live = row < V;
#pragma unroll
            for (int t = 0; t < T; ++t) nbn[t] = live ? nbr[row * T + t] : -1;
        } else {
            const int64_t row = mt * 32 + lrow;
            const bool live = row < V;
#pragma unroll
            for (int t = 0; t < T; ++t) nb[t] = live ? nbr[row * T + t] : -1;
        }

        f32x16_t acc[CB];
#pragma unroll
        for (int j = 0; j < CB; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[j][r] = 0.f;

        u32x4_t ar[PT][KG][AW];
        auto load_tap = [&](int t, int slot) {
            const int u = nb[t];
            const int64_t rr = u >= 0 ? u : 0;
            const char *base = reinterpret_cast<const char *>(in) + rr * C_IN * IN_ESZ;
#pragma unroll
            for (int g = 0; g < KG; ++g)
#pragma unroll
                for (int w = 0; w < AW; ++w)
                    ar[slot][g][w] = *reinterpret_cast<const u32x4_t *>(
                        base + (g * KGE + khalf * (KGE / 2)) * IN_ESZ + w * 16);
        };
        auto compute_tap = [&](int t, int slot) {
            const bool pres = nb[t] >= 0;
#pragma unroll
            for (int g = 0; g < KG; ++g) {
                u32x4_t a;
                if (CM == 1) {
                    const u32x4_t x0 = ar[slot][g][0], x1 = ar[slot][g][1];
                    a[0] = bf16_bits(__uint_as_float(x0[0])) | (bf16_bits(__uint_as_float(x0[1])) << 16);
                    a[1] = bf16_bits(__uint_as_float(x0[2])) | (bf16_bits(__uint_as_float(x0[3])) << 16);
                    a[2] = bf16_bits(__uint_as_float(x1[0])) | (bf16_bits(__uint_as_float(x1[1])) << 16);
                    a[3] = bf16_bits(__uint_as_float(x1[2])) | (bf16_bits(__uint_as_float(x1[3])) << 16);
                } else {
                    a = ar[slot][g][0];
                }
                if (!pres) a = u32x4_t{0u, 0u, 0u, 0u};
                const int kb = (t * C_IN + g * KGE) * WESZ + khalf * 16;
                u32x4_t b[CB];
#pragma unroll
                for (int j = 0; j < CB; ++j)
                    b[j] = *reinterpret_cast<const u32x4_t *>(wlds + (j * 32 + lrow) * KSTRIDE + kb);
                if (BF16) {
#pragma unroll
                    for (int j = 0; j < CB; ++j)
                        acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                                         __builtin_bit_cast(bf16x8_t, b[j]), acc[j],
                                                                         0, 0, 0);
                } else {
                    // independent accumulators innermost, so consecutive MFMAs do not wait on each other
#pragma unroll
                    for (int c = 0; c < 4; ++c)
#pragma unroll
                        for (int j = 0; j < CB; ++j)
                            acc[j] = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a[c]),
                                                                          __uint_as_float(b[j][c]), acc[j], 0, 0, 0);
                }
            }
        };
#pragma unroll
        for (int t = 0; t < PT && t < T; ++t) load_tap(t, t);
        // The fences keep the scheduler from hoisting later taps' loads above
        // earlier taps' MFMAs, which would hold all T taps in registers.
#pragma unroll
        for (int t = 0; t < T; ++t) {
            __builtin_amdgcn_sched_barrier(0);
            compute_tap(t, t % PT);
            if (t + PT < T) load_tap(t + PT, t % PT);
        }
        __builtin_amdgcn_sched_barrier(0);

#pragma unroll
        for (int j = 0; j < CB; ++j) {
            const int col = col_base + j * 32 + lrow;
            const float bc = bias ? bias[col] : 0.f;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int64_t orow = mt * 32 + 8 * (r >> 2) + 4 * khalf + (r & 3);
                if (orow < V) {
                    const float y = acc[j][r] + bc;
                    if (OUT_BF16)
                        reinterpret_cast<uint16_t *>(out)[orow * C_out + col] = (uint16_t)bf16_bits(y);
                    else
                        reinterpret_cast<float *>(out)[orow * C_out + col] = y;
                }
            }
        }
    }
}

// ---------------------------------------------------------------------------
// k_conv_rs: bf16 rows and weights, weights resident in registers.
//
// A gather in MFMA operand layout puts 32 different rows in one 64-lane load
// (each lane 16 bytes), which the address unit serves one lane per cycle.
// Here the gathered rows travel instead by direct-to-LDS loads in row order
// (consecutive lanes read consecutive 16-byte chunks of a row, so a load is
// a few full cache lines), into a two-tile LDS ring; the MFMA operand is
// then read from LDS.  Each of the four wavefronts owns 32 output columns
// and keeps their whole K x 32 weight slice in registers for the life of
// the workgroup, so the weights cost neither LDS bandwidth nor address-unit
// cycles after the prologue; with C_out = 64 two wavefronts share a column
// group and split the rows.
//
// Per tile of MT rows (MT = 32 * 4 / (C_out / 32)):
//   top:   wait for this tile's loads, barrier
//          issue the next tile's row loads (addresses from its neighbour
//          block, already in LDS) and the neighbour block of the tile after
//          that
//   body:  T taps x C_in/16 k-groups of ds_read + MFMA 32x32x16
//   store: bias, fp32 or bf16
// A missing neighbour (index -1) and the rows past V of the last tile read
// a zero row.  16-byte chunk c of tile row r sits at chunk c ^ (r % 8) of
// the row's LDS slot (and weight row n likewise with n % 8), so that the
// 32-row operand reads spread over the LDS banks.
namespace rs {
typedef __attribute__((address_space(3))) void lds_void;

__device__ __forceinline__ void dma16(const void *src, char *lds_wave_base) {
    __builtin_amdgcn_global_load_lds(src, (lds_void *)lds_wave_base, 16, 0, 0);
}

// Wait for every outstanding memory operation of this wavefront (the
// direct-to-LDS loads included), then the workgroup barrier.  The memory
// clobber keeps the compiler from moving LDS accesses across it.
__device__ __forceinline__ void drain_and_barrier() { asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory"); }
}  // namespace rs

template <int C_IN, int C_OUT, int T>
struct RsShape {
    static constexpr int NW = 4;
    static constexpr int NCG = C_OUT / 32;                 // column groups
    static constexpr int NRG = NW / NCG;                   // row groups
    static constexpr int MT = 32 * NRG;                    // rows per tile
    static constexpr int K = T * C_IN;
    static constexpr int KG = K / 16;                      // k-groups (one MFMA each)
    static constexpr int GPT = C_IN / 16;                  // k-groups per tap
    static constexpr int CPR = C_IN / 8;                   // 16-byte chunks per row
    static constexpr int SLICE = MT * CPR;                 // chunks of one tap
    static constexpr int TILE = T * SLICE;                 // chunks of one tile
    static constexpr int TILE_BYTES = TILE * 16;
    static constexpr int ADMA = TILE / (64 * NW);          // row loads per wavefront per tile
    static constexpr int NB_INTS = MT * T;                 // neighbour block of a tile
    static constexpr int NB_DMA = (NB_INTS * 4 + 1023) / 1024;
    static constexpr int NB_BYTES = NB_DMA * 1024;
    static constexpr int WCPR = K / 8;                     // chunks per weight row
    static constexpr int W_ROWS_ROUND = (2 * TILE_BYTES) / (WCPR * 16) < C_OUT ? (2 * TILE_BYTES) / (WCPR * 16) : C_OUT;
    static constexpr int W_ROUNDS = C_OUT / W_ROWS_ROUND;
    static constexpr int W_DMA = W_ROWS_ROUND * WCPR / (64 * NW);  // weight loads per wavefront per round
    static constexpr int LDS = 2 * TILE_BYTES + 2 * NB_BYTES;
    static constexpr int PD = GPT >= 8 ? 1 : 2;            // operand read-ahead, in taps
    static constexpr int DPT = ADMA / T;                   // row loads issued per tap
    static_assert(DPT * T == ADMA, "row loads per tap");
    static_assert(NCG * NRG == NW, "column groups");
    static_assert(TILE % (64 * NW) == 0, "tile loads");
    static_assert(CPR >= 8 && WCPR % 8 == 0, "swizzle");
    static_assert(NB_DMA <= NW && NB_INTS % 4 == 0, "neighbour block");
    static_assert(W_ROWS_ROUND % 32 == 0 && C_OUT % W_ROWS_ROUND == 0, "weight rounds");
    static_assert((W_ROWS_ROUND * WCPR) % (64 * NW) == 0, "weight loads");
    static_assert(LDS <= 160 * 1024, "LDS");
};

template <bool OUT_BF16, int T, int C_IN, int C_OUT>
__global__ __launch_bounds__(256) void k_conv_rs(const uint16_t *__restrict__ in, const uint16_t *__restrict__ w,
                                                 const float *__restrict__ bias, void *__restrict__ out,
                                                 const int32_t *__restrict__ nbr, int64_t nbr_ints,
                                                 const int32_t *__restrict__ counters,
                                                 const uint16_t *__restrict__ zero_row) {
    using S = RsShape<C_IN, C_OUT, T>;
    extern __shared__ __attribute__((aligned(16))) char lds[];
    auto abuf = [&](int b) { return lds + b * S::TILE_BYTES; };                      // row tiles
    auto nbuf = [&](int b) { return lds + 2 * S::TILE_BYTES + b * S::NB_BYTES; };    // neighbour blocks

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int l32 = lane & 31;
    const int h = lane >> 5;
    const int cg = wave % S::NCG;
    const int rg = wave / S::NCG;
    const int64_t V = counters[CNT_V];
    const int64_t n_tiles = (V + S::MT - 1) / S::MT;
    const int64_t tile0 = blockIdx.x;
    const int64_t tstride = gridDim.x;
    if (tile0 >= n_tiles) return;  // uniform over the workgroup

    // Neighbour block of tile k -> nbuf(b): NB_INTS contiguous ints, one
    // 1 KB load per wavefront for the first NB_DMA wavefronts; chunks past
    // the block or past the buffer re-read an in-bounds chunk.
    auto load_nbr = [&](int64_t k, int b) {
        if (wave < S::NB_DMA) {
            const int64_t j = (int64_t)wave * 64 + lane;
            const int64_t last = (nbr_ints / 4 - 1) * 4;  // last whole 16-byte chunk of the table
            int64_t at = k * S::NB_INTS + 4 * j;
            if (4 * j >= S::NB_INTS) at = k * S::NB_INTS;
            if (at > last) at = last;
            rs::dma16(nbr + at, nbuf(b) + wave * 1024);
        }
    };
    // Rows of tile k -> abuf(b).  A wavefront's ADMA loads are issued DPT
    // per tap between the MFMAs of the current tile, so that the address
    // unit drains them while the matrix cores work; the neighbour indices of
    // tap t's loads are read from nbuf(b) one tap earlier (a direct-to-LDS
    // load is not reordered with LDS reads, so reading an index right before
    // its load would wait out the LDS latency).
    auto read_nb = [&](int b, int t, int *u) {
        const int32_t *nb = reinterpret_cast<const int32_t *>(nbuf(b));
#pragma unroll
        for (int i = 0; i < S::DPT; ++i) {
            const int q = (wave * S::ADMA + t * S::DPT + i) * 64 + lane;
            const int tt = q / S::SLICE;
            const int r = (q - tt * S::SLICE) / S::CPR;
            u[i] = nb[r * T + tt];
        }
    };
    auto issue_rows = [&](int64_t k, int b, int t, const int *u) {
        const int rows_left = (int)(V - k * S::MT < S::MT ? V - k * S::MT : S::MT);
#pragma unroll
        for (int i = 0; i < S::DPT; ++i) {
            const int a = t * S::DPT + i;
            const int q = (wave * S::ADMA + a) * 64 + lane;
            const int tt = q / S::SLICE;
            const int pr = q - tt * S::SLICE;
            const int r = pr / S::CPR;
            const int cs = pr - r * S::CPR;
            const bool ok = r < rows_left && u[i] >= 0;
            const uint16_t *src = ok ? in + (int64_t)u[i] * C_IN + ((cs ^ (r & 7)) * 8) : zero_row;
            rs::dma16(src, abuf(b) + (wave * S::ADMA + a) * 1024);
        }
    };

    // Prologue: weights -> registers, in rounds of W_ROWS_ROUND rows staged
    // in the (still unused) tile buffers; the first tile's neighbour block
    // travels with the first round.
    u32x4_t bw[S::KG];
#pragma unroll
    for (int rd = 0; rd < S::W_ROUNDS; ++rd) {
        const int n0 = rd * S::W_ROWS_ROUND;
#pragma unroll
        for (int a = 0; a < S::W_DMA; ++a) {
            const int q = (wave * S::W_DMA + a) * 64 + lane;
            const int r = q / S::WCPR;
            const int cs = q - r * S::WCPR;
            const int n = n0 + r;
            rs::dma16(w + (int64_t)n * S::K + ((cs ^ (n & 7)) * 8), lds + (wave * S::W_DMA + a) * 1024);
        }
        if (rd == 0) load_nbr(tile0, 0);
        rs::drain_and_barrier();
        if (cg * 32 >= n0 && cg * 32 < n0 + S::W_ROWS_ROUND) {
            const int n = cg * 32 + l32;
            const char *row = lds + (n - n0) * S::WCPR * 16;
#pragma unroll
            for (int kg = 0; kg < S::KG; ++kg)
                bw[kg] = *reinterpret_cast<const u32x4_t *>(row + (((2 * kg + h) ^ (n & 7)) * 16));
        }
        rs::drain_and_barrier();
    }
#pragma unroll
    for (int t = 0; t < T; ++t) {
        int u[S::DPT];
        read_nb(0, t, u);
        issue_rows(tile0, 0, t, u);
    }
    if (tile0 + tstride < n_tiles) load_nbr(tile0 + tstride, 1);

    const float bcol = bias ? bias[cg * 32 + l32] : 0.f;
    int b = 0;
    for (int64_t k = tile0; k < n_tiles; k += tstride, b ^= 1) {
        rs::drain_and_barrier();
        const bool next = k + tstride < n_tiles;
        int ucur[S::DPT], unext[S::DPT];
        if (next) read_nb(b ^ 1, 0, ucur);
        if (k + 2 * tstride < n_tiles) load_nbr(k + 2 * tstride, b);

        f32x16_t acc0, acc1;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            acc0[i] = 0.f;
            acc1[i] = 0.f;
        }
        const int r = rg * 32 + l32;
        const char *arow = abuf(b) + r * S::CPR * 16;
        // Operand fragments are read PD taps ahead of their MFMAs (one
        // wavefront per SIMD: nothing else hides the LDS latency).
        constexpr int PD = S::PD;
        u32x4_t af[PD + 1][S::GPT];
        auto read_tap = [&](int t, int slot) {
#pragma unroll
            for (int g = 0; g < S::GPT; ++g)
                af[slot][g] = *reinterpret_cast<const u32x4_t *>(arow + t * S::SLICE * 16 + (((2 * g + h) ^ (r & 7)) * 16));
        };
#pragma unroll
        for (int t = 0; t < PD && t < T; ++t) read_tap(t, t);
#pragma unroll
        for (int t = 0; t < T; ++t) {
            if (next) {
                issue_rows(k + tstride, b ^ 1, t, ucur);
                if (t + 1 < T) read_nb(b ^ 1, t + 1, unext);
#pragma unroll
                for (int i = 0; i < S::DPT; ++i) ucur[i] = unext[i];
            }
            if (t + PD < T) read_tap(t + PD, (t + PD) % (PD + 1));
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int g = 0; g < S::GPT; ++g) {
                const bf16x8_t a = __builtin_bit_cast(bf16x8_t, af[t % (PD + 1)][g]);
                const bf16x8_t bb = __builtin_bit_cast(bf16x8_t, bw[t * S::GPT + g]);
                if (t & 1)
                    acc1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, bb, acc1, 0, 0, 0);
                else
                    acc0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, bb, acc0, 0, 0, 0);
            }
            __builtin_amdgcn_sched_barrier(0);
        }
        const int col = cg * 32 + l32;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            const int64_t orow = k * S::MT + rg * 32 + 8 * (i >> 2) + 4 * h + (i & 3);
            if (orow < V) {
                const float y = acc0[i] + acc1[i] + bcol;
                if (OUT_BF16)
                    reinterpret_cast<uint16_t *>(out)[orow * C_OUT + col] = (uint16_t)bf16_bits(y);
                else
                    reinterpret_cast<float *>(out)[orow * C_OUT + col] = y;
            }
        }
    }
}

// Any storage/compute combination, one thread per output element.
template <bool IN_BF16, bool BF16, bool OUT_BF16>
__global__ __launch_bounds__(256) void k_conv_generic(const void *__restrict__ in, int C_in,
                                                      const void *__restrict__ wv, int C_out, int T,
                                                      const float *__restrict__ bias, void *__restrict__ out,
                                                      const int32_t *__restrict__ nbr,
                                                      const int32_t *__restrict__ counters) {
    const int64_t V = counters[CNT_V];
    const int64_t n = V * C_out;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n; e += stride) {
        const int64_t v = e / C_out;
        const int o = (int)(e - v * C_out);
        float acc = bias ? bias[o] : 0.f;
        for (int t = 0; t < T; ++t) {
            const int u = nbr[v * T + t];
            if (u < 0) continue;
            const int64_t xb = (int64_t)u * C_in;
            const int64_t wb = ((int64_t)o * T + t) * C_in;
            for (int i = 0; i < C_in; ++i) {
                float xv = IN_BF16 ? bf16_to_f32(reinterpret_cast<const uint16_t *>(in)[xb + i])
                                   : reinterpret_cast<const float *>(in)[xb + i];
                float wvv;
                if (BF16) {
                    xv = __uint_as_float(bf16_bits(xv) << 16);
                    wvv = bf16_to_f32(reinterpret_cast<const uint16_t *>(wv)[wb + i]);
                } else {
                    wvv = reinterpret_cast<const float *>(wv)[wb + i];
                }
                acc = fmaf(xv, wvv, acc);
            }
        }
        if (OUT_BF16)
            reinterpret_cast<uint16_t *>(out)[e] = (uint16_t)bf16_bits(acc);
        else
            reinterpret_cast<float *>(out)[e] = acc;
    }
}

template <int CM, bool OUT_BF16, int BM, int BN, int WR, int WC, int P>
hipError_t launch_mfma(lattice *L, const void *in, int C_in, const void *w, int C_out, const float *bias, void *out) {
    constexpr int NT = (BM / WR) * (BN / WC) * 64;
    constexpr int LDS = 2 * (BM + BN) * kRowBytes + BM * kMaxTaps * 4;
    constexpr int PER_CU = (160 * 1024) / LDS < 4 ? (160 * 1024) / LDS : 4;  // resident workgroups per CU
    const int64_t tiles = ((L->max_vertices + BM - 1) / BM) * (C_out / BN);
    int64_t grid = (int64_t)L->cu_count * PER_CU;
    if (grid > tiles) grid = tiles;
    if (grid < 1) grid = 1;
    hipLaunchKernelGGL((k_conv_mfma<CM, OUT_BF16, BM, BN, WR, WC, P>), dim3((unsigned)grid), dim3(NT), 0, L->stream,
                       in, C_in, w, C_out, L->T, bias, out, L->nbr, L->counters);
    return hipGetLastError();
}

template <int CM, bool OUT_BF16>
hipError_t launch_mfma_n(lattice *L, const void *in, int C_in, const void *w, int C_out, const float *bias,
                         void *out) {
    constexpr int P = CM == 1 ? 2 : 3;
    // fp32: 64 x 64 tiles, four workgroups per CU (the fp32 MFMA is slow enough
    // that four waves per SIMD keep it busy; small tiles shorten the tail)
    if (CM == 0) return launch_mfma<CM, OUT_BF16, 64, 64, 32, 32, 2>(L, in, C_in, w, C_out, bias, out);
    if (C_out % 128 == 0) return launch_mfma<CM, OUT_BF16, 128, 128, 64, 64, P>(L, in, C_in, w, C_out, bias, out);
    return launch_mfma<CM, OUT_BF16, 128, 64, 32, 64, P>(L, in, C_in, w, C_out, bias, out);
}

template <bool IN_BF16, bool BF16, bool OUT_BF16>
hipError_t launch_generic(lattice *L, const void *in, int C_in, const void *w, int C_out, const float *bias,
                          void *out) {
    const unsigned grid = grid_for(L->max_vertices * (int64_t)C_out, 256, L->cu_count, 8);
    hipLaunchKernelGGL((k_conv_generic<IN_BF16, BF16, OUT_BF16>), dim3(grid), dim3(256), 0, L->stream, in, C_in, w,
                       C_out, L->T, bias, out, L->nbr, L->counters);
    return hipGetLastError();
}

constexpr int kWsMaxLds = 152 * 1024;  // weight slice budget of one workgroup

template <int CM, bool OUT_BF16, int T, int C_IN, int CB, int PT>
hipError_t launch_ws(lattice *L, const void *in, const void *w, int C_out, const float *bias, void *out) {
    constexpr int BN = 32 * CB;
    constexpr int WESZ = CM != 0 ? 2 : 4;
    constexpr int LDS = BN * (T * C_IN * WESZ + 16);
    static_assert(LDS <= kWsMaxLds, "weight slice exceeds LDS");
    auto kern = k_conv_ws<CM, OUT_BF16, T, C_IN, CB, PT>;
    static bool attr_set = false;
    if (!attr_set) {
        hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                           hipFuncAttributeMaxDynamicSharedMemorySize, LDS);
        if (e != hipSuccess) return e;
        attr_set = true;
    }
    const int n_nt = C_out / BN;
    const int64_t tiles = ((L->max_vertices + 31) / 32) * n_nt;
    int64_t grid = (int64_t)L->cu_count;
    grid = ((grid + n_nt - 1) / n_nt) * n_nt;  // whole groups of N slices
    const int64_t need = ((tiles + 7) / 8 + n_nt - 1) / n_nt * n_nt;  // no more workgroups than 8-wave groups of tiles
    if (grid > need) grid = need < n_nt ? n_nt : need;
    hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(512), LDS, L->stream, in, w, C_out, bias, out, L->nbr,
                       L->counters);
    return hipGetLastError();
}

template <bool OUT_BF16, int T, int C_IN, int C_OUT>
hipError_t launch_rs(lattice *L, const void *in, const void *w, const float *bias, void *out) {
    using S = RsShape<C_IN, C_OUT, T>;
    auto kern = k_conv_rs<OUT_BF16, T, C_IN, C_OUT>;
    static bool attr_set = false;
    if (!attr_set) {
        hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                           hipFuncAttributeMaxDynamicSharedMemorySize, S::LDS);
        if (e != hipSuccess) return e;
        attr_set = true;
    }
    const int per_cu = (160 * 1024) / S::LDS < 2 ? 1 : 2;
    const int64_t tiles = (L->max_vertices + S::MT - 1) / S::MT;
    int64_t grid = (int64_t)L->cu_count * per_cu;
    if (grid > tiles) grid = tiles;
    if (grid < 1) grid = 1;
    hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(256), S::LDS, L->stream,
                       reinterpret_cast<const uint16_t *>(in), reinterpret_cast<const uint16_t *>(w), bias, out,
                       L->nbr, L->max_vertices * (int64_t)L->T, L->counters, L->zero_row);
    return hipGetLastError();
}

// Register-stationary dispatch (bf16 rows and weights); false when the shape
// is not one it is built for.
template <bool OUT_BF16>
bool try_rs(lattice *L, const void *in, int C_in, const void *w, int C_out, const float *bias, void *out,
            hipError_t *err) {
    const int T = L->T;
    if (T == 9 && C_in == 64 && C_out == 64) *err = launch_rs<OUT_BF16, 9, 64, 64>(L, in, w, bias, out);
    else if (T == 9 && C_in == 64 && C_out == 128) *err = launch_rs<OUT_BF16, 9, 64, 128>(L, in, w, bias, out);
    else if (T == 9 && C_in == 128 && C_out == 128) *err = launch_rs<OUT_BF16, 9, 128, 128>(L, in, w, bias, out);
    else if (T == 11 && C_in == 64 && C_out == 128) *err = launch_rs<OUT_BF16, 11, 64, 128>(L, in, w, bias, out);
    else return false;
    return true;
}

// Weight-stationary dispatch for the shapes it covers; returns false when
// the shape is not covered (the caller falls back to k_conv_mfma).
template <bool OUT_BF16>
bool try_ws(lattice *L, const void *in, bool in_bf16, int C_in, const void *w, int C_out, bool bf16,
            const float *bias, void *out, hipError_t *err) {
#define WS(CM, TT, CI, CBV, PTV)                                                                   \
    do {                                                                                           \
        *err = launch_ws<CM, OUT_BF16, TT, CI, CBV, PTV>(L, in, w, C_out, bias, out);             \
        return true;                                                                               \
    } while (0)
    const int T = L->T;
    if (T != 9 && T != 11) return false;
    if (!bf16) return false;  // fp32 runs on the LDS-tiled kernel
    if (bf16 && in_bf16) {
        if (C_in == 64) {
            if (C_out % 128 == 0) {
                if (T == 9) WS(2, 9, 64, 4, 2);
                WS(2, 11, 64, 2, 3);
            }
            if (C_out % 64 == 0) {
                if (T == 9) WS(2, 9, 64, 2, 3);
                WS(2, 11, 64, 2, 3);
            }
        }
        if (C_in == 128 && C_out % 64 == 0) {
            if (T == 9) WS(2, 9, 128, 2, 2);
            WS(2, 11, 128, 1, 2);
        }
        return false;
    }
    if (bf16 && !in_bf16 && C_in == 64 && C_out % 64 == 0) {
        if (T == 9) WS(1, 9, 64, 2, 2);
        WS(1, 11, 64, 2, 2);
    }
    return false;
#undef WS
}

template <bool OUT_BF16>
hipError_t dispatch_out(lattice *L, const void *in, lattice_dtype in_dt, int C_in, const void *w, int C_out,
                        lattice_dtype dt, const float *bias, void *out) {
    const bool in_bf16 = in_dt == LATTICE_BF16;
    const bool bf16 = dt == LATTICE_BF16;
    const bool aligned = ((reinterpret_cast<uintptr_t>(in) & 15) == 0) && ((reinterpret_cast<uintptr_t>(w) & 15) == 0);
    const int path = L->conv_path;
    if (aligned && (path == LATTICE_CONV_AUTO || path == LATTICE_CONV_RS) && bf16 && in_bf16) {
        hipError_t err = hipSuccess;
        if (try_rs<OUT_BF16>(L, in, C_in, w, C_out, bias, out, &err)) return err;
    }
    if (aligned && path != LATTICE_CONV_TILED) {
        hipError_t err = hipSuccess;
        if (try_ws<OUT_BF16>(L, in, in_bf16, C_in, w, C_out, bf16, bias, out, &err)) return err;
    }
    if (aligned && C_out % 64 == 0) {
        if (!bf16 && !in_bf16 && C_in % 32 == 0)
            return launch_mfma_n<0, OUT_BF16>(L, in, C_in, w, C_out, bias, out);
        if (bf16 && !in_bf16 && C_in % 64 == 0)
            return launch_mfma_n<1, OUT_BF16>(L, in, C_in, w, C_out, bias, out);
        if (bf16 && in_bf16 && C_in % 64 == 0)
            return launch_mfma_n<2, OUT_BF16>(L, in, C_in, w, C_out, bias, out);
    }
    if (in_bf16)
        return bf16 ? launch_generic<true, true, OUT_BF16>(L, in, C_in, w, C_out, bias, out)
                    : launch_generic<true, false, OUT_BF16>(L, in, C_in, w, C_out, bias, out);
    return bf16 ? launch_generic<false, true, OUT_BF16>(L, in, C_in, w, C_out, bias, out)
                : launch_generic<false, false, OUT_BF16>(L, in, C_in, w, C_out, bias, out);
}

}  // namespace

hipError_t launch_conv(lattice *L, const void *in, lattice_dtype in_dt, int C_in, const void *w, int C_out,
                       lattice_dtype dt, const float *bias, void *out, lattice_dtype out_dt) {
    return out_dt == LATTICE_BF16 ? dispatch_out<true>(L, in, in_dt, C_in, w, C_out, dt, bias, out)
                                  : dispatch_out<false>(L, in, in_dt, C_in, w, C_out, dt, bias, out);
}
