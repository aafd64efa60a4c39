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
// k_conv_any: MFMA over any channel counts and alignments (e.g. 8 -> 16),
// with the operands gathered element by element.
#include <type_traits>

#include "internal.h"

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

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
// k_conv_rs: weights resident in registers, rows gathered into LDS.
//
// A gather in MFMA operand layout puts 32 different rows in one 64-lane load
// (each lane 16 bytes); measured on this chip such loads move about a third
// of what row-order loads of the same rows do.  Here the gathered rows
// travel by direct-to-LDS loads in row order (consecutive lanes read
// consecutive 16-byte chunks of a row) into a two-tile LDS ring, and the
// MFMA operands are read from LDS.  A wavefront owns 32 output columns and
// 1/KS of the K = T C_in reduction, and keeps that K/KS x 32 weight slice in
// registers for the life of the workgroup: after the prologue the weights
// cost neither LDS bandwidth nor address-unit cycles.  With KS = 2 the two
// halves are added through LDS at the end of each tile.
//
// Operand groups: a lane's 16-byte chunk (2g + h) of a row (h = lane / 32)
// is the k-slice h of group g: bf16, 8 channels of one MFMA 32x32x16; fp32,
// channels 8g + 4h + i, the k = h operand of MFMA 32x32x2 number i of the
// group.  The weights are held in the same order.
//
// Per tile of MT rows:
//   top:   wait for this tile's loads, barrier; issue the neighbour block
//          of the tile after next and the next tile's row loads (addresses
//          from its neighbour block, already in LDS)
//   body:  T steps of KG/T operand groups (ds_read + MFMA)
//   store: (KS = 2: partial sums through LDS) bias, fp32 or bf16
// A missing neighbour (index -1) and the rows past V of the last tile read
// a zero row.  16-byte chunks of tile rows (and of staged weight rows) are
// XOR-swizzled by row (rs::swz), so that the 32-row operand reads spread
// over the LDS banks.
namespace rs {
typedef __attribute__((address_space(3))) void lds_void;

__device__ __forceinline__ void dma16(const void *src, char *lds_wave_base) {
    __builtin_amdgcn_global_load_lds(src, (lds_void *)lds_wave_base, 16, 0, 0);
}

// Wait for every outstanding memory operation of this wavefront (the
// direct-to-LDS loads included), then the workgroup barrier.  The memory
// clobber keeps the compiler from moving LDS accesses across it.
__device__ __forceinline__ void drain_and_barrier() { asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// XOR key of row r for rows of P 16-byte chunks in LDS: chunk c of row r is
// stored at chunk c ^ swz<P>(r).  Sixteen consecutive rows of a 16-lane
// read pass then hit sixteen different 16-byte bank groups (256 bytes of
// banks): with P a multiple of 16 the key is r mod 16; with P an odd
// multiple of 8, rows alternate between the two bank halves and the key is
// (r / 2) mod 8.
template <int P>
__device__ __forceinline__ int swz(int r) {
    static_assert(P % 16 == 0 || (P % 8 == 0 && (P / 8) % 2 == 1), "row pitch");
    return P % 16 == 0 ? (r & 15) : ((r >> 1) & 7);
}

// Barrier after this wavefront's LDS operations (no wait on global memory).
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// 4 x 4 transpose within each quad of lanes: on entry lane j of a quad
// holds element (i, j) in v[i]; on return it holds element (j, i) in v[i].
// Two exchange rounds (quad_perm 2,3,0,1 then 1,0,3,2).
__device__ __forceinline__ void quad_transpose(float *v) {
    const int j = threadIdx.x & 3;
    int x[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) x[i] = __builtin_amdgcn_mov_dpp(__float_as_int(v[i]), 0x4E, 0xF, 0xF, false);
    if (j < 2) {
        v[2] = __int_as_float(x[0]);
        v[3] = __int_as_float(x[1]);
    } else {
        v[0] = __int_as_float(x[2]);
        v[1] = __int_as_float(x[3]);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) x[i] = __builtin_amdgcn_mov_dpp(__float_as_int(v[i]), 0xB1, 0xF, 0xF, false);
    if ((j & 1) == 0) {
        v[1] = __int_as_float(x[0]);
        v[3] = __int_as_float(x[2]);
    } else {
        v[0] = __int_as_float(x[1]);
        v[2] = __int_as_float(x[3]);
    }
}

// Store a 32 x 32 MFMA accumulator block (lane l: column l % 32, register i:
// row 8 (i / 4) + 4 (l / 32) + i % 4) plus bias: after a quad transpose a
// lane holds four consecutive columns of one row, stored as one 16-byte
// (fp32) or 8-byte (bf16) write.  Rows at or past V are not written.
template <bool OUT_BF16>
__device__ __forceinline__ void store_block(f32x16_t acc, float bias_col, void *out, int64_t row0, int col0,
                                            int C_out, int64_t V) {
    const int lane = threadIdx.x & 63;
    const int j = lane & 3;
    const int h = lane >> 5;
    const int c = col0 + (lane & 31) - j;  // first of the lane's four columns
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        float v[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) v[i] = acc[4 * q + i] + bias_col;  // bias of column (lane & 31)
        quad_transpose(v);
        // v[i] now: row 8q + 4h + j, column c + i (the bias moved with it)
        const int64_t row = row0 + 8 * q + 4 * h + j;
        if (row < V) {
            if (OUT_BF16) {
                uint2 pk;
                pk.x = bf16_bits(v[0]) | (bf16_bits(v[1]) << 16);
                pk.y = bf16_bits(v[2]) | (bf16_bits(v[3]) << 16);
                *reinterpret_cast<uint2 *>(reinterpret_cast<uint16_t *>(out) + row * C_out + c) = pk;
            } else {
                *reinterpret_cast<float4 *>(reinterpret_cast<float *>(out) + row * C_out + c) =
                    make_float4(v[0], v[1], v[2], v[3]);
            }
        }
    }
}

// Wait until at most N vector memory operations of this wavefront are
// outstanding (and its LDS operations are done), then the barrier.
template <int N>
__device__ __forceinline__ void wait_vm_barrier() {
    static_assert(N >= 0 && N < 64, "vmcnt");
    asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(N) : "memory");
}
}  // namespace rs

template <bool BF16, int C_IN, int C_OUT, int T, int KS>
struct RsShape {
    static constexpr int NW = 4;
    static constexpr int ESZ = BF16 ? 2 : 4;
    static constexpr int NCG = C_OUT / 32;                 // column groups
    static constexpr int NRG = NW / (NCG * KS);            // row groups
    static constexpr int MT = 32 * NRG;                    // rows per tile
    static constexpr int K = T * C_IN;
    static constexpr int CPR = C_IN * ESZ / 16;            // 16-byte chunks per row
    static constexpr int GPT = CPR / 2;                    // operand groups per tap
    static constexpr int KG = T * GPT;                     // operand groups
    static constexpr int KGW = KG / KS;                    // operand groups per wavefront
    static constexpr int GPS = KGW / T;                    // groups per step
    static constexpr int SLICE = MT * CPR;                 // chunks of one tap
    static constexpr int TILE = T * SLICE;                 // chunks of one tile
    static constexpr int TILE_BYTES = TILE * 16;
    static constexpr int ADMA = TILE / (64 * NW);          // row loads per wavefront per tile
    static constexpr int NB_INTS = MT * T;                 // neighbour block of a tile
    static constexpr int NB_DMA = (NB_INTS * 4 + 1023) / 1024;
    static constexpr int NB_BYTES = NB_DMA * 1024;
    static constexpr int RED_BYTES = KS > 1 ? NCG * NRG * 16 * 64 * 4 : 0;  // partial sums (in the tile's buffer)
    static constexpr int WCPR = K * ESZ / 16;              // chunks per weight row
    static constexpr int W_ROWS_ROUND = (2 * TILE_BYTES) / (WCPR * 16) < C_OUT ? (2 * TILE_BYTES) / (WCPR * 16) : C_OUT;
    static constexpr int W_ROUNDS = C_OUT / W_ROWS_ROUND;
    static constexpr int W_DMA = W_ROWS_ROUND * WCPR / (64 * NW);  // weight loads per wavefront per round
    static constexpr int LDS = 2 * TILE_BYTES + 2 * NB_BYTES;
    // Two workgroups per CU (two wavefronts per SIMD, at most 256 registers
    // each) when both fit in LDS and the weight slice leaves room: the
    // second workgroup's loads are in flight while the first multiplies.
    static constexpr int WPE = (2 * LDS <= 160 * 1024 && KGW * 4 <= 160) ? 2 : 1;
    static constexpr int PD = (GPS >= 8 || WPE == 2) ? 1 : 2;  // operand read-ahead, in steps
    static_assert(NCG * NRG * KS == NW && NRG >= 1, "wavefront roles");
    static_assert(KG % KS == 0 && KGW % T == 0, "groups per step");
    static_assert(TILE % (64 * NW) == 0, "tile loads");
    static_assert(CPR >= 8 && WCPR % 8 == 0, "swizzle");
    static_assert(NB_DMA <= NW && NB_INTS % 4 == 0, "neighbour block");
    static_assert(W_ROWS_ROUND % 32 == 0 && C_OUT % W_ROWS_ROUND == 0, "weight rounds");
    static_assert((W_ROWS_ROUND * WCPR) % (64 * NW) == 0, "weight loads");
    static_assert(LDS <= 160 * 1024, "LDS");
    static_assert(RED_BYTES <= TILE_BYTES, "partial sums fit in a tile buffer");
};

template <bool BF16, bool OUT_BF16, int T, int C_IN, int C_OUT, int KS>
__global__ __launch_bounds__(256, (RsShape<BF16, C_IN, C_OUT, T, KS>::WPE)) void k_conv_rs(const void *__restrict__ in_, const void *__restrict__ w_,
                                                 const float *__restrict__ bias, void *__restrict__ out,
                                                 const int32_t *__restrict__ nbr, int64_t nbr_ints,
                                                 const int32_t *__restrict__ counters,
                                                 const uint16_t *__restrict__ zero_row) {
    using S = RsShape<BF16, C_IN, C_OUT, T, KS>;
    const char *in = reinterpret_cast<const char *>(in_);
    const char *w = reinterpret_cast<const char *>(w_);
    extern __shared__ __attribute__((aligned(16))) char lds[];
    auto abuf = [&](int b) { return lds + b * S::TILE_BYTES; };                      // row tiles
    auto nbuf = [&](int b) { return lds + 2 * S::TILE_BYTES + b * S::NB_BYTES; };    // neighbour blocks

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int l32 = lane & 31;
    const int h = lane >> 5;
    const int cg = wave % S::NCG;
    const int rg = (wave / S::NCG) % S::NRG;
    const int ks = KS == 1 ? 0 : wave / (S::NCG * S::NRG);
    const int64_t V = counters[CNT_V];
    const int64_t n_tiles = (V + S::MT - 1) / S::MT;
    const int64_t tile0 = blockIdx.x;
    const int64_t tstride = gridDim.x;
    if (tile0 >= n_tiles) return;  // uniform over the workgroup

    // The bias is in a register before the first direct-to-LDS load: its
    // first use would otherwise make the compiler wait for every load issued
    // before it.
    float bcol = bias ? bias[cg * 32 + l32] : 0.f;
    asm volatile("s_waitcnt vmcnt(0)" : "+v"(bcol));

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
    // Row load a (0 .. ADMA-1) of this wavefront for tile k into abuf(b):
    // the neighbour index first (from nbuf(b)), then the load.
    auto row_nb = [&](int b, int a) {
        const int q = (wave * S::ADMA + a) * 64 + lane;
        const int t = q / S::SLICE;
        const int r = (q - t * S::SLICE) / S::CPR;
        return reinterpret_cast<const int32_t *>(nbuf(b))[r * T + t];
    };
    auto row_load = [&](int64_t k, int b, int a, int u) {
        const int q = (wave * S::ADMA + a) * 64 + lane;
        const int t = q / S::SLICE;
        const int pr = q - t * S::SLICE;
        const int r = pr / S::CPR;
        const int cs = pr - r * S::CPR;
        const bool ok = r < V - k * S::MT && u >= 0;
        const void *src = ok ? (const void *)(in + ((int64_t)u * C_IN * S::ESZ + ((cs ^ rs::swz<S::CPR>(r)) * 16)))
                             : (const void *)zero_row;
        rs::dma16(src, abuf(b) + (wave * S::ADMA + a) * 1024);
    };

    // Prologue: weights -> registers, in rounds of W_ROWS_ROUND rows staged
    // in the (still unused) tile buffers; the first tile's neighbour block
    // travels with the first round.
    u32x4_t bw[S::KGW];
#pragma unroll
    for (int rd = 0; rd < S::W_ROUNDS; ++rd) {
        const int n0 = rd * S::W_ROWS_ROUND;
#pragma unroll
        for (int a = 0; a < S::W_DMA; ++a) {
            const int q = (wave * S::W_DMA + a) * 64 + lane;
            const int r = q / S::WCPR;
            const int cs = q - r * S::WCPR;
            const int n = n0 + r;
            rs::dma16(w + ((int64_t)n * S::WCPR + (cs ^ rs::swz<S::WCPR>(n))) * 16, lds + (wave * S::W_DMA + a) * 1024);
        }
        if (rd == 0) load_nbr(tile0, 0);
        rs::drain_and_barrier();
        if (cg * 32 >= n0 && cg * 32 < n0 + S::W_ROWS_ROUND) {
            const int n = cg * 32 + l32;
            const char *row = lds + (n - n0) * S::WCPR * 16;
#pragma unroll
            for (int kk = 0; kk < S::KGW; ++kk) {
                const int kg = ks * S::KGW + kk;
                bw[kk] = *reinterpret_cast<const u32x4_t *>(row + (((2 * kg + h) ^ rs::swz<S::WCPR>(n)) * 16));
            }
        }
        rs::drain_and_barrier();
    }
#pragma unroll
    for (int a = 0; a < S::ADMA; ++a) row_load(tile0, 0, a, row_nb(0, a));
    if (tile0 + tstride < n_tiles) load_nbr(tile0 + tstride, 1);

    const int r = rg * 32 + l32;
    int b = 0;
    for (int64_t k = tile0; k < n_tiles; k += tstride, b ^= 1) {
        rs::drain_and_barrier();
        const bool next = k + tstride < n_tiles;
        if (k + 2 * tstride < n_tiles) load_nbr(k + 2 * tstride, b);
        // the next tile's row loads: all neighbour indices first (a
        // direct-to-LDS load is not reordered with LDS reads, so alternating
        // them would serialise both), then the loads
        if (next) {
            int u[S::ADMA];
#pragma unroll
            for (int i = 0; i < S::ADMA; ++i) u[i] = row_nb(b ^ 1, i);
#pragma unroll
            for (int i = 0; i < S::ADMA; ++i) row_load(k + tstride, b ^ 1, i, u[i]);
        }

        f32x16_t acc0, acc1;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            acc0[i] = 0.f;
            acc1[i] = 0.f;
        }
        const char *arow = abuf(b) + r * S::CPR * 16;
        // operand group kk of this wavefront: tap kg / GPT, group kg % GPT
        auto read_group = [&](int kk) {
            const int kg = ks * S::KGW + kk;
            const int t = kg / S::GPT;
            const int g = kg - t * S::GPT;
            return *reinterpret_cast<const u32x4_t *>(arow + t * S::SLICE * 16 + (((2 * g + h) ^ rs::swz<S::CPR>(r)) * 16));
        };
        // Operand groups are read PD steps ahead of their MFMAs (with one
        // wavefront per SIMD nothing else hides the LDS latency; with two,
        // the other one does).  With PD = 1 a single set of registers: group
        // g of step st+1 is read as soon as the MFMAs of group g of step st
        // are issued.
        constexpr int PD = S::PD;
        constexpr int NSETS = PD == 1 ? 1 : PD + 1;
        u32x4_t af[NSETS][S::GPS];
#pragma unroll
        for (int st = 0; st < PD && st < T; ++st)
#pragma unroll
            for (int g = 0; g < S::GPS; ++g) af[st][g] = read_group(st * S::GPS + g);
#pragma unroll
        for (int st = 0; st < T; ++st) {
            if (PD != 1 && st + PD < T) {
#pragma unroll
                for (int g = 0; g < S::GPS; ++g) af[(st + PD) % (PD + 1)][g] = read_group((st + PD) * S::GPS + g);
            }
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int g = 0; g < S::GPS; ++g) {
                const u32x4_t a = af[PD == 1 ? 0 : st % (PD + 1)][g];
                const u32x4_t bb = bw[st * S::GPS + g];
                if (BF16) {
                    if (g & 1)
                        acc1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                                       __builtin_bit_cast(bf16x8_t, bb), acc1, 0, 0, 0);
                    else
                        acc0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                                       __builtin_bit_cast(bf16x8_t, bb), acc0, 0, 0, 0);
                } else {
#pragma unroll
                    for (int c = 0; c < 4; ++c) {
                        if (c & 1)
                            acc1 = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a[c]), __uint_as_float(bb[c]),
                                                                        acc1, 0, 0, 0);
                        else
                            acc0 = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a[c]), __uint_as_float(bb[c]),
                                                                        acc0, 0, 0, 0);
                    }
                }
                if (PD == 1 && st + 1 < T) af[0][g] = read_group((st + 1) * S::GPS + g);
            }
            __builtin_amdgcn_sched_barrier(0);
        }
#pragma unroll
        for (int i = 0; i < 16; ++i) acc0[i] += acc1[i];
        if (KS > 1) {
            // the second K half adds its partial sums through LDS, in this
            // tile's row buffer once every wavefront has read its operands
            // (the next loads into it are issued after the next top barrier)
            rs::lds_barrier();
            float *slot = reinterpret_cast<float *>(abuf(b)) + ((cg * S::NRG + rg) * 16) * 64;
            if (ks == 1) {
#pragma unroll
                for (int i = 0; i < 16; ++i) slot[i * 64 + lane] = acc0[i];
            }
            rs::lds_barrier();
            if (ks == 0) {
#pragma unroll
                for (int i = 0; i < 16; ++i) acc0[i] += slot[i * 64 + lane];
            }
        }
        if (KS == 1 || ks == 0) rs::store_block<OUT_BF16>(acc0, bcol, out, k * S::MT + rg * 32, cg * 32, C_OUT, V);
    }
}

// ---------------------------------------------------------------------------
// k_conv_ring: register-resident weights like k_conv_rs, with the gathered
// rows streamed through a ring of T tap slices (slot t holds tap t of some
// tile) instead of two whole tiles, so that fp32 rows (and T = 11) fit in
// LDS.  A slice is MT rows x C_in channels; each wavefront issues DPS
// direct-to-LDS loads per slice.  At the top of slice j (tile i, tap t):
//   wait until slices j .. j+PD are in LDS, barrier (slot of j-1 is free)
//   t = 0: store tile i-1 and clear the accumulators
//   t = 1: load the neighbour block of tile i+2 into tile i's buffer, whose
//   last reads (the indices of tap T-1, at t = 0) the barrier has retired
//   in every wavefront
//   read the operands of slice j+PD; MFMAs of slice j, with the loads of
//   slice j+T-1 (tap t-1 of tile i+1; for t = 0 the last tap of tile i)
//   into the freed slot issued between them.
// The wait is a vmcnt bound: loads complete in issue order, so "at most N
// loads newer than slice j+PD outstanding" means j+PD has landed; N counts
// the DMA groups issued after it (and the neighbour-block load where that
// is newer: for 2 <= t <= T-1-PD).  Stores are not counted: a store still
// in flight only makes the wait longer.  Loads past the last tile read the
// zero row so that every wavefront issues the same number of loads per slice.
//
// fp32: a lane's 16-byte chunk (2g + h) of a row holds channels 8g + 4h + i,
// i = 0..3, the k = h operand of MFMA 32x32x2 number i of the group; the
// weights are held in the same permutation.
template <bool BF16, int C_IN, int C_OUT, int T>
struct RingShape {
    static constexpr int NW = 4;
    static constexpr int ESZ = BF16 ? 2 : 4;
    static constexpr int NCG = C_OUT / 32;
    static constexpr int NRG = NW / NCG;
    static constexpr int MT = 32 * NRG;
    static constexpr int K = T * C_IN;
    static constexpr int CPR = C_IN * ESZ / 16;            // 16-byte chunks per row
    static constexpr int GPT = CPR / 2;                    // 32-byte operand groups per tap
    static constexpr int SLICE_BYTES = MT * CPR * 16;
    static constexpr int DPS = SLICE_BYTES / (1024 * NW);  // loads per wavefront per slice
    static constexpr int RING_BYTES = T * SLICE_BYTES;
    static constexpr int NB_INTS = MT * T;
    static constexpr int NB_BYTES = NW * 1024;             // one 1 KB load per wavefront
    static constexpr int PD = BF16 ? 2 : 1;                // operand read-ahead, in slices
    static constexpr int WCPR = K * ESZ / 16;              // chunks per weight row
    static constexpr int W_ROWS_ROUND = (RING_BYTES / (WCPR * 16)) / 32 * 32 < C_OUT
                                            ? (RING_BYTES / (WCPR * 16)) / 32 * 32 : C_OUT;
    static constexpr int W_ROUNDS = C_OUT / W_ROWS_ROUND;
    static constexpr int W_DMA = W_ROWS_ROUND * WCPR / (64 * NW);
    static constexpr int LDS = RING_BYTES + 2 * NB_BYTES;
    static_assert(NCG * NRG == NW && MT >= 32, "column groups");
    static_assert(SLICE_BYTES % (1024 * NW) == 0, "slice loads");
    static_assert(CPR >= 8 && WCPR % 8 == 0, "swizzle");
    static_assert(NB_INTS * 4 <= NB_BYTES && NB_INTS % 4 == 0, "neighbour block");
    static_assert(W_ROWS_ROUND >= 32 && C_OUT % W_ROWS_ROUND == 0, "weight rounds");
    static_assert((W_ROWS_ROUND * WCPR) % (64 * NW) == 0, "weight loads");
    static_assert(T - 2 - PD >= 1, "ring depth");
    static_assert(GPT % DPS == 0, "loads spread over the operand groups");
    static_assert(LDS <= 160 * 1024, "LDS");
};

template <bool BF16, bool OUT_BF16, int T, int C_IN, int C_OUT>
__global__ __launch_bounds__(256) void k_conv_ring(const void *__restrict__ in_, const void *__restrict__ w_,
                                                   const float *__restrict__ bias, void *__restrict__ out,
                                                   const int32_t *__restrict__ nbr, int64_t nbr_ints,
                                                   const int32_t *__restrict__ counters,
                                                   const uint16_t *__restrict__ zero_row) {
    using S = RingShape<BF16, C_IN, C_OUT, T>;
    const char *in = reinterpret_cast<const char *>(in_);
    const char *w = reinterpret_cast<const char *>(w_);
    extern __shared__ __attribute__((aligned(16))) char lds[];
    auto slot = [&](int t) { return lds + t * S::SLICE_BYTES; };
    auto nbuf = [&](int b) { return lds + S::RING_BYTES + b * S::NB_BYTES; };

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

    // neighbour block of tile k (may be past the last tile) -> nbuf(b)
    auto load_nbr = [&](int64_t k, int b) {
        const int64_t last = (nbr_ints / 4 - 1) * 4;
        const int64_t j = (int64_t)wave * 64 + lane;
        int64_t at = k * S::NB_INTS + 4 * j;
        if (4 * j >= S::NB_INTS) at = k * S::NB_INTS;
        if (at > last) at = last;
        rs::dma16(nbr + at, nbuf(b) + wave * 1024);
    };
    // tap t of tile k -> slot(t): the DPS neighbour indices of this
    // wavefront's loads (from nbuf(b)), then one load at a time
    auto slice_nb = [&](int b, int t, int *u) {
        const int32_t *nb = reinterpret_cast<const int32_t *>(nbuf(b));
#pragma unroll
        for (int i = 0; i < S::DPS; ++i) {
            const int q = (wave * S::DPS + i) * 64 + lane;
            u[i] = nb[(q / S::CPR) * T + t];
        }
    };
    auto slice_load = [&](int64_t k, int t, int i, int u) {
        const int q = (wave * S::DPS + i) * 64 + lane;
        const int r = q / S::CPR;
        const int cs = q - r * S::CPR;
        const bool ok = r < V - k * S::MT && u >= 0;
        const void *src = ok ? (const void *)(in + ((int64_t)u * C_IN * S::ESZ + ((cs ^ rs::swz<S::CPR>(r)) * 16)))
                             : (const void *)zero_row;
        rs::dma16(src, slot(t) + (wave * S::DPS + i) * 1024);
    };
    auto load_slice = [&](int64_t k, int b, int t) {
        int u[S::DPS];
        slice_nb(b, t, u);
#pragma unroll
        for (int i = 0; i < S::DPS; ++i) slice_load(k, t, i, u[i]);
    };

    // The bias is in a register before the first direct-to-LDS load: its
    // first use would otherwise make the compiler wait for every load issued
    // before it.
    float bcol = bias ? bias[cg * 32 + l32] : 0.f;
    asm volatile("s_waitcnt vmcnt(0)" : "+v"(bcol));

    // Prologue: weights -> registers (rounds staged in the ring), the first
    // two neighbour blocks, then taps 0..T-2 of the first tile.
    u32x4_t bw[T * S::GPT];
#pragma unroll
    for (int rd = 0; rd < S::W_ROUNDS; ++rd) {
        const int n0 = rd * S::W_ROWS_ROUND;
#pragma unroll
        for (int a = 0; a < S::W_DMA; ++a) {
            const int q = (wave * S::W_DMA + a) * 64 + lane;
            const int r = q / S::WCPR;
            const int cs = q - r * S::WCPR;
            const int n = n0 + r;
            rs::dma16(w + ((int64_t)n * S::WCPR + (cs ^ rs::swz<S::WCPR>(n))) * 16, lds + (wave * S::W_DMA + a) * 1024);
        }
        if (rd == 0) {
            load_nbr(tile0, 0);
            load_nbr(tile0 + tstride, 1);
        }
        rs::drain_and_barrier();
        if (cg * 32 >= n0 && cg * 32 < n0 + S::W_ROWS_ROUND) {
            const int n = cg * 32 + l32;
            const char *row = lds + (n - n0) * S::WCPR * 16;
#pragma unroll
            for (int kg = 0; kg < T * S::GPT; ++kg)
                bw[kg] = *reinterpret_cast<const u32x4_t *>(row + (((2 * kg + h) ^ rs::swz<S::WCPR>(n)) * 16));
        }
        rs::drain_and_barrier();
    }
#pragma unroll
    for (int t = 0; t < T - 1; ++t) load_slice(tile0, 0, t);

    const int r = rg * 32 + l32;
    // Operands: with PD = 1 one set of registers, group g of slice j+1
    // read as soon as the MFMAs of group g of slice j are issued; with PD = 2
    // a ring of PD + 1 sets.
    constexpr int NSETS = S::PD == 1 ? 1 : S::PD + 1;
    u32x4_t af[NSETS][S::GPT];
    auto read_group = [&](int t, int sl, int g) {
        const char *arow = slot(t) + r * S::CPR * 16;
        af[sl][g] = *reinterpret_cast<const u32x4_t *>(arow + (((2 * g + h) ^ rs::swz<S::CPR>(r)) * 16));
    };
    auto read_slice = [&](int t, int sl) {
#pragma unroll
        for (int g = 0; g < S::GPT; ++g) read_group(t, sl, g);
    };
    f32x16_t acc0, acc1;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
        acc0[i] = 0.f;
        acc1[i] = 0.f;
    }
    auto store_tile = [&](int64_t k) {
#pragma unroll
        for (int i = 0; i < 16; ++i) acc0[i] += acc1[i];
        rs::store_block<OUT_BF16>(acc0, bcol, out, k * S::MT + rg * 32, cg * 32, C_OUT, V);
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            acc0[i] = 0.f;
            acc1[i] = 0.f;
        }
    };

    int b = 0;  // parity of tile i's neighbour buffer
    bool first = true;
    for (int64_t k = tile0; k < n_tiles; k += tstride, b ^= 1) {
#pragma unroll
        for (int t = 0; t < T; ++t) {
            // wait for slices j .. j+PD (see above), then the barrier
            if (t >= 2 && t <= T - 1 - S::PD)
                rs::wait_vm_barrier<(T - 2 - S::PD) * S::DPS + 1>();
            else
                rs::wait_vm_barrier<(T - 2 - S::PD) * S::DPS>();
            // slice j+T-1: tap T-1 of this tile (t = 0) or tap t-1 of the next
            const int64_t lk = t == 0 ? k : k + tstride;
            const int lt = t == 0 ? T - 1 : t - 1;
            int u[S::DPS];
            slice_nb(t == 0 ? b : b ^ 1, lt, u);
            if (t == 0) {
                if (!first) store_tile(k - tstride);
                first = false;
            }
            if (t == 1) load_nbr(k + 2 * tstride, b);
            if (k == tile0 && t == 0) {
#pragma unroll
                for (int p = 0; p < S::PD; ++p) read_slice(p, p);
            }
            // operands of slice j + PD (tap (t + PD) mod T), PD = 2
            if (S::PD != 1) read_slice((t + S::PD) % T, (t + S::PD) % (S::PD + 1));
            __builtin_amdgcn_sched_barrier(0);
            // MFMAs of slice j, with the DPS loads of slice j+T-1 spread
            // between them so that the address unit works while they run
            constexpr int GPL = S::GPT / S::DPS;  // groups per load
#pragma unroll
            for (int g = 0; g < S::GPT; ++g) {
                const u32x4_t a = af[S::PD == 1 ? 0 : t % (S::PD + 1)][g];
                const u32x4_t bb = bw[t * S::GPT + g];
                if (BF16) {
                    if (g & 1)
                        acc1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                                       __builtin_bit_cast(bf16x8_t, bb), acc1, 0, 0, 0);
                    else
                        acc0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                                       __builtin_bit_cast(bf16x8_t, bb), acc0, 0, 0, 0);
                } else {
#pragma unroll
                    for (int c = 0; c < 4; ++c) {
                        if (c & 1)
                            acc1 = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a[c]), __uint_as_float(bb[c]),
                                                                        acc1, 0, 0, 0);
                        else
                            acc0 = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a[c]), __uint_as_float(bb[c]),
                                                                        acc0, 0, 0, 0);
                    }
                }
                if (S::PD == 1) read_group((t + 1) % T, 0, g);  // operands of slice j+1
                if (g % GPL == GPL - 1) slice_load(lk, lt, g / GPL, u[g / GPL]);
                __builtin_amdgcn_sched_barrier(0);
            }
        }
        // The operands of the next tile's first PD slices were read into
        // af[(t' + T) % (PD + 1)]; the tile body expects them at af[t'].
        if (S::PD != 1 && T % (S::PD + 1) != 0) {
            u32x4_t tmp[S::PD + 1][S::GPT];
#pragma unroll
            for (int p = 0; p < S::PD; ++p)
#pragma unroll
                for (int g = 0; g < S::GPT; ++g) tmp[p][g] = af[(p + T) % (S::PD + 1)][g];
#pragma unroll
            for (int p = 0; p < S::PD; ++p)
#pragma unroll
                for (int g = 0; g < S::GPT; ++g) af[p][g] = tmp[p][g];
        }
    }
    store_tile(n_tiles - 1 - (n_tiles - 1 - tile0) % tstride);
}

// Any shape and any storage/compute combination on MFMA: the fallback for
// channel counts the tilings above do not cover (C_in or C_out not a
// multiple of 32 / 64, e.g. 8 -> 16), and for operands that are not 16-byte
// aligned.  The product is the same Y = Z W^T over the flattened
// K = T C_in: a workgroup of WM x WN wavefronts owns a (32 WM) x (32 WN)
// output tile, each wavefront one 32 x 32 MFMA block.  K is walked in
// chunks of KC = 64: every thread gathers its share of the chunk's
// elements one by one (k -> tap k / C_in, channel k % C_in, through the
// tile's neighbour indices staged in LDS), zero past K, past C_out and for
// absent neighbours, converts them to the MFMA operand type and writes them
// to LDS; the next chunk's elements are loaded into registers while the
// current one is multiplied.  Operands in LDS are K-contiguous rows padded
// by 16 bytes (an odd number of 16-byte units per row).  MMA_BF16: rows
// rounded to bf16 (nearest even; bf16-stored rows are taken as they are)
// and bf16 weights, MFMA 32x32x16; otherwise fp32 rows and weights, MFMA
// 32x32x2 (lane half h holds k = 8 g + 4 h + c in component c of a group
// g, as in k_conv_mfma).
constexpr int kAnyKC = 64;

template <bool IN_BF16, bool MMA_BF16, bool OUT_BF16, int WM, int WN>
__global__ __launch_bounds__(WM * WN * 64) void k_conv_any(const void *__restrict__ in, int C_in,
                                                           const void *__restrict__ wv, int C_out, int T,
                                                           const float *__restrict__ bias, void *__restrict__ out,
                                                           const int32_t *__restrict__ nbr,
                                                           const int32_t *__restrict__ counters) {
    constexpr int NT = WM * WN * 64;
    constexpr int BM = 32 * WM;
    constexpr int BN = 32 * WN;
    constexpr int ESZ = MMA_BF16 ? 2 : 4;          // operand element in LDS
    constexpr int PITCH = kAnyKC * ESZ + 16;       // bytes per LDS row
    constexpr int A_PER = BM * kAnyKC / NT;        // A elements per thread per chunk
    constexpr int B_PER = BN * kAnyKC / NT;
    static_assert(A_PER * NT == BM * kAnyKC && B_PER * NT == BN * kAnyKC, "chunk split");
    typedef typename std::conditional<MMA_BF16, uint16_t, float>::type op_t;

    __shared__ __attribute__((aligned(16))) char As[BM * PITCH];
    __shared__ __attribute__((aligned(16))) char Bs[BN * PITCH];
    __shared__ int32_t nbr_s[BM * kMaxTaps];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave / WN;
    const int wn = wave % WN;
    const int lrow = lane & 31;
    const int h = lane >> 5;
    const int64_t V = counters[CNT_V];
    const int64_t n_mt = (V + BM - 1) / BM;
    const int n_nt = (C_out + BN - 1) / BN;
    const int64_t ntiles = n_mt * n_nt;
    const int64_t K = (int64_t)T * C_in;
    const int64_t NQ = (K + kAnyKC - 1) / kAnyKC;

    // Lane kk of every wavefront owns K column kk of each chunk (rows
    // wave, wave + NW, ...), so the tap and channel of its elements are
    // worked out once per chunk, and a wavefront reads 64 consecutive
    // elements of one row.
    constexpr int NW = WM * WN;
    const int kk = lane;
    auto a_elem = [&](int r, int t, int i, bool in_k) -> op_t {
        float x = 0.f;
        uint16_t xb = 0;
        const int u = in_k ? nbr_s[r * T + t] : -1;
        if (u >= 0) {
            if (IN_BF16) {
                xb = reinterpret_cast<const uint16_t *>(in)[(int64_t)u * C_in + i];
                x = bf16_to_f32(xb);
            } else {
                x = reinterpret_cast<const float *>(in)[(int64_t)u * C_in + i];
                xb = (uint16_t)bf16_bits(x);
            }
        }
        if constexpr (MMA_BF16) return xb;
        else return x;
    };

    for (int64_t tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
        const int64_t row_base = (tile / n_nt) * BM;
        const int col_base = (int)(tile % n_nt) * BN;
        for (int i = tid; i < BM * T; i += NT) {
            const int64_t e = row_base * T + i;
            nbr_s[i] = (e < V * T) ? nbr[e] : -1;
        }
        __syncthreads();

        op_t ar[A_PER], br[B_PER];
        auto load_chunk = [&](int64_t q) {
            const int64_t k = q * kAnyKC + kk;
            const bool in_k = k < K;
            const int t = in_k ? (int)(k / C_in) : 0;
            const int i = in_k ? (int)(k - (int64_t)t * C_in) : 0;
#pragma unroll
            for (int j = 0; j < A_PER; ++j) ar[j] = a_elem(wave + j * NW, t, i, in_k);
#pragma unroll
            for (int j = 0; j < B_PER; ++j) {
                const int col = col_base + wave + j * NW;
                br[j] = (in_k && col < C_out) ? reinterpret_cast<const op_t *>(wv)[(int64_t)col * K + k] : op_t(0);
            }
        };
        auto store_chunk = [&]() {
#pragma unroll
            for (int j = 0; j < A_PER; ++j)
                *reinterpret_cast<op_t *>(As + (wave + j * NW) * PITCH + kk * ESZ) = ar[j];
#pragma unroll
            for (int j = 0; j < B_PER; ++j)
                *reinterpret_cast<op_t *>(Bs + (wave + j * NW) * PITCH + kk * ESZ) = br[j];
        };

        f32x16_t acc;
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[r] = 0.f;
        const char *arow = As + (wm * 32 + lrow) * PITCH;
        const char *brow = Bs + (wn * 32 + lrow) * PITCH;

        load_chunk(0);
        for (int64_t q = 0; q < NQ; ++q) {
            store_chunk();
            __syncthreads();
            if (q + 1 < NQ) load_chunk(q + 1);
            if constexpr (MMA_BF16) {
#pragma unroll
                for (int g = 0; g < kAnyKC / 16; ++g) {
                    const u32x4_t a = *reinterpret_cast<const u32x4_t *>(arow + (16 * g + 8 * h) * 2);
                    const u32x4_t b = *reinterpret_cast<const u32x4_t *>(brow + (16 * g + 8 * h) * 2);
                    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                                  __builtin_bit_cast(bf16x8_t, b), acc, 0, 0, 0);
                }
            } else {
#pragma unroll
                for (int g = 0; g < kAnyKC / 8; ++g) {
                    const u32x4_t a = *reinterpret_cast<const u32x4_t *>(arow + (8 * g + 4 * h) * 4);
                    const u32x4_t b = *reinterpret_cast<const u32x4_t *>(brow + (8 * g + 4 * h) * 4);
#pragma unroll
                    for (int c = 0; c < 4; ++c)
                        acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a[c]), __uint_as_float(b[c]), acc,
                                                                   0, 0, 0);
                }
            }
            __syncthreads();  // LDS is rewritten by the next chunk
        }

        // register r of lane l: row 8 (r / 4) + 4 (l / 32) + r % 4, column l % 32
        const int col = col_base + wn * 32 + lrow;
        if (col < C_out) {
            const float bc = bias ? bias[col] : 0.f;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int64_t row = row_base + wm * 32 + 8 * (r >> 2) + 4 * h + (r & 3);
                if (row < V) {
                    const float y = acc[r] + bc;
                    if (OUT_BF16)
                        reinterpret_cast<uint16_t *>(out)[row * C_out + col] = (uint16_t)bf16_bits(y);
                    else
                        reinterpret_cast<float *>(out)[row * C_out + col] = y;
                }
            }
        }
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
    if constexpr (CM == 0) {
        return launch_mfma<CM, OUT_BF16, 64, 64, 32, 32, 2>(L, in, C_in, w, C_out, bias, out);
    } else {
        if (C_out % 128 == 0) return launch_mfma<CM, OUT_BF16, 128, 128, 64, 64, P>(L, in, C_in, w, C_out, bias, out);
        return launch_mfma<CM, OUT_BF16, 128, 64, 32, 64, P>(L, in, C_in, w, C_out, bias, out);
    }
}

template <bool IN_BF16, bool MMA_BF16, bool OUT_BF16>
hipError_t launch_any(lattice *L, const void *in, int C_in, const void *w, int C_out, const float *bias, void *out) {
    if (L->T > kMaxTaps) return hipErrorInvalidValue;
    // C_out <= 32: 128 x 32 tiles (four wavefronts along M); else 64 x 64
    auto go = [&](auto kern, int bm, int bn) {
        const int64_t tiles = ((L->max_vertices + bm - 1) / bm) * ((C_out + bn - 1) / bn);
        int64_t grid = (int64_t)L->cu_count * 4;
        if (grid > tiles) grid = tiles;
        if (grid < 1) grid = 1;
        hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(256), 0, L->stream, in, C_in, w, C_out, L->T, bias, out,
                           L->nbr, L->counters);
        return hipGetLastError();
    };
    if (C_out <= 32) return go(k_conv_any<IN_BF16, MMA_BF16, OUT_BF16, 4, 1>, 128, 32);
    return go(k_conv_any<IN_BF16, MMA_BF16, OUT_BF16, 2, 2>, 64, 64);
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

template <bool BF16, bool OUT_BF16, int T, int C_IN, int C_OUT, int KS>
hipError_t launch_rs(lattice *L, const void *in, const void *w, const float *bias, void *out) {
    using S = RsShape<BF16, C_IN, C_OUT, T, KS>;
    auto kern = k_conv_rs<BF16, OUT_BF16, T, C_IN, C_OUT, KS>;
    static bool attr_set = false;
    if (!attr_set) {
        hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                           hipFuncAttributeMaxDynamicSharedMemorySize, S::LDS);
        if (e != hipSuccess) return e;
        attr_set = true;
    }
    const int per_cu = S::WPE;
    const int64_t tiles = (L->max_vertices + S::MT - 1) / S::MT;
    int64_t grid = (int64_t)L->cu_count * per_cu;
    if (grid > tiles) grid = tiles;
    if (grid < 1) grid = 1;
    hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(256), S::LDS, L->stream, in, w, bias, out, L->nbr,
                       L->max_vertices * (int64_t)L->T, L->counters, L->zero_row);
    return hipGetLastError();
}

template <bool BF16, bool OUT_BF16, int T, int C_IN, int C_OUT>
hipError_t launch_ring(lattice *L, const void *in, const void *w, const float *bias, void *out) {
    using S = RingShape<BF16, C_IN, C_OUT, T>;
    auto kern = k_conv_ring<BF16, OUT_BF16, T, C_IN, C_OUT>;
    static bool attr_set = false;
    if (!attr_set) {
        hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                           hipFuncAttributeMaxDynamicSharedMemorySize, S::LDS);
        if (e != hipSuccess) return e;
        attr_set = true;
    }
    const int64_t tiles = (L->max_vertices + S::MT - 1) / S::MT;
    int64_t grid = (int64_t)L->cu_count;
    if (grid > tiles) grid = tiles;
    if (grid < 1) grid = 1;
    hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(256), S::LDS, L->stream, in, w, bias, out, L->nbr,
                       L->max_vertices * (int64_t)L->T, L->counters, L->zero_row);
    return hipGetLastError();
}

// Register-stationary dispatch (bf16 rows and weights); false when the shape
// is not one it is built for.
template <bool OUT_BF16>
bool try_rs(lattice *L, const void *in, int C_in, const void *w, int C_out, const float *bias, void *out,
            hipError_t *err) {
    const int T = L->T;
    if (T == 11 && C_in == 64 && C_out == 64) *err = launch_ring<true, OUT_BF16, 11, 64, 64>(L, in, w, bias, out);
    else if (T == 9 && C_in == 64 && C_out == 64) *err = launch_rs<true, OUT_BF16, 9, 64, 64, 2>(L, in, w, bias, out);
    else if (T == 9 && C_in == 64 && C_out == 128) *err = launch_rs<true, OUT_BF16, 9, 64, 128, 1>(L, in, w, bias, out);
    else if (T == 9 && C_in == 128 && C_out == 128) *err = launch_rs<true, OUT_BF16, 9, 128, 128, 1>(L, in, w, bias, out);
    else if (T == 11 && C_in == 64 && C_out == 128) *err = launch_rs<true, OUT_BF16, 11, 64, 128, 1>(L, in, w, bias, out);
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
    // the register-resident kernels store four columns at once (16 bytes of
    // fp32, 8 of bf16); the others store single elements
    const bool out_vec = (reinterpret_cast<uintptr_t>(out) & (OUT_BF16 ? 7 : 15)) == 0;
    const int path = L->conv_path;
    if (aligned && out_vec && (path == LATTICE_CONV_AUTO || path == LATTICE_CONV_RS) && bf16 && in_bf16) {
        hipError_t err = hipSuccess;
        if (try_rs<OUT_BF16>(L, in, C_in, w, C_out, bias, out, &err)) return err;
    }
    // fp32 64 -> 64: the register-resident kernel (K split over two
    // wavefronts) only on request; the LDS-tiled kernel is faster there
    if (aligned && out_vec && path == LATTICE_CONV_RS && !bf16 && !in_bf16 && L->T == 9 && C_in == 64 && C_out == 64)
        return launch_rs<false, OUT_BF16, 9, 64, 64, 2>(L, in, w, bias, out);
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
        return bf16 ? launch_any<true, true, OUT_BF16>(L, in, C_in, w, C_out, bias, out)
                    : launch_any<true, false, OUT_BF16>(L, in, C_in, w, C_out, bias, out);
    return bf16 ? launch_any<false, true, OUT_BF16>(L, in, C_in, w, C_out, bias, out)
                : launch_any<false, false, OUT_BF16>(L, in, C_in, w, C_out, bias, out);
}

}  // namespace

hipError_t launch_conv(lattice *L, const void *in, lattice_dtype in_dt, int C_in, const void *w, int C_out,
                       lattice_dtype dt, const float *bias, void *out, lattice_dtype out_dt) {
    return out_dt == LATTICE_BF16 ? dispatch_out<true>(L, in, in_dt, C_in, w, C_out, dt, bias, out)
                                  : dispatch_out<false>(L, in, in_dt, C_in, w, C_out, dt, bias, out);
}
