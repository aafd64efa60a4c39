// Internal declarations shared by the host API (lattice.hip) and the kernel
// translation units (splat.hip, neighbors.hip, conv.hip, slice.hip, deform.hip,
// backward.hip, distribute.hip).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "lattice.h"

// Device status bits, OR-ed into counters[CNT_STATUS] by kernels.
// ST_CLOUDS: a batched lattice's batch ids exceed the range the group
// normalisation keeps per-cloud statistics for.
enum : int { ST_CAPACITY = 1, ST_RANGE = 2, ST_CLOUDS = 4 };
// Slots of the device counter array.
// CNT_SPLIT and CNT_ROWS count the vertices whose pair list the splat gather
// cuts into parts, and those parts.
// CNT_SLOTS is the number of hash slots the last numbering recorded in
// vslot (every occupied slot of the table, one per vertex), which the next
// splat empties instead of the whole table.
// CNT_NB is 1 + the largest batch id of a batched lattice's vertices (set by
// the distribute operation, for its per-cloud statistics).
enum : int {
    CNT_V = 0, CNT_STATUS = 1, CNT_E = 2, CNT_SPLIT = 3, CNT_ROWS = 4, CNT_SLOTS = 5, CNT_NB = 6, CNT_WORDS = 8
};

// A vertex's pair list longer than kPart pairs is cut into parts of kPart
// pairs (the splat's gather work units, also used by the distribute op); the
// splat's numbering records the split vertices and their part rows.
constexpr int kPart = 32;

// A pair-list entry is (point and slot, weight): the point index p in bits
// 0..27 (lattice_create bounds max_points by 2^28) and in bits 28..30 the
// slot k (the remainder) of the vertex in p's simplex, so that a consumer
// finds the pair's per-point record (p (d+1) + k) without a search.
constexpr int kListPointBits = 28;
constexpr int32_t kListPointMask = (1 << kListPointBits) - 1;
__host__ __device__ __forceinline__ int32_t list_entry(int64_t p, int k) {
    return (int32_t)p | (k << kListPointBits);
}
__host__ __device__ __forceinline__ int32_t list_point(int32_t x) { return x & kListPointMask; }
__host__ __device__ __forceinline__ int list_slot(int32_t x) { return x >> kListPointBits; }

// Packed 64-bit vertex key: 16 bits per coordinate c_0..c_{d-1}, each stored
// as c + KEY_BIAS (so a field is never 0 for |c| <= KEY_MAX), and for d <= 3
// the batch id in bits 48..63.  c_d is implied by the zero sum.  0 marks an
// empty hash slot.
constexpr int KEY_BIAS = 32768;
constexpr int KEY_MAX = 32767;

struct HEntry;  // hash table entry (keys.h)

// fp32 -> bf16 bits, round to nearest with ties to even (NaN stays a quiet NaN).
__device__ __forceinline__ uint32_t bf16_bits(float f) {
    const uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (u >> 16) | 0x40u;
    return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}

__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

struct lattice_timer {
    double ms = 0.0;    // summed elapsed time of read event pairs
    int64_t count = 0;  // number of read event pairs
};

struct lattice {
    int d = 0;
    int T = 0;
    double alpha = 0.0;
    float sigma[LATTICE_MAX_D] = {0};
    float factors[LATTICE_MAX_D] = {0};  // alpha / (sigma_{j-1} sqrt(j(j+1))), fp32
    float inv_dp1 = 0.f;                 // fp32(1/(d+1))
    int64_t max_points = 0;
    int64_t cap = 0;          // hash slots, power of two
    int64_t max_vertices = 0; // min((d+1) max_points, cap)
    int device = 0;
    hipStream_t stream = nullptr;

    HEntry *tab = nullptr;      // [cap] hash table {key, pair count, vertex index}
    uint32_t *occ = nullptr;    // [(cap + 31) / 32] occupancy bit of each slot (set by the numbering, for lookups)
    uint64_t *vkeys = nullptr;  // [max_vertices] packed key of each vertex
    int32_t *vslot = nullptr;   // [max_vertices] hash slot of each vertex (what the next splat empties)
    bool full_clear = true;     // the table may hold keys vslot does not list: empty all of it
    int32_t *blk = nullptr;     // [scan_blocks_max()][4] per-block sums of the numbering scan
    int32_t *vinfo = nullptr;   // [max_vertices][2] (offset, count) of the vertex's pair list
    // Long pair lists are gathered in parts (splat.hip); at most
    // split_rows_max() parts and split vertices per splat.
    int32_t *split = nullptr;   // [rows_max][3] (vertex, first part row, parts) per split vertex
    int32_t *rowmap = nullptr;  // [rows_max] split index of each part row
    int32_t *partrec = nullptr; // [rows_max][2] (list offset of its first pair, pairs) of each part row
    float *pweight = nullptr;   // [rows_max] partial weight sums
    float *partial = nullptr;   // [rows_max][partial_cols] partial feature sums, grown on demand
    int64_t partial_cols = 0;
    // Backward scratch (backward.hip), grown on the first call that needs more.
    void *wflip = nullptr;      // flipped, transposed conv weights [C_in][T][C_out]
    int64_t wflip_bytes = 0;
    float *wgpart = nullptr;    // weight-gradient partials [chunks][C_out][T][C_in], then bias partials
    int64_t wgpart_floats = 0;
    void *dfb = nullptr;        // DeformSlice backward: per-point records and partials (deform_bwd.hip)
    int64_t dfb_bytes = 0;
    void *pnb = nullptr;        // Distribute + PointNet backward: row records and partials (distribute.hip)
    int64_t pnb_bytes = 0;
    // Cross-lattice neighbour tables [max_vertices][T], built on demand:
    // xtab[0] when this lattice is the coarse output of a downsampling,
    // xtab[1] when it is the fine output of an upsampling.  Each remembers
    // the source lattice and both splat generations it was built for.
    int32_t *xtab[2] = {nullptr, nullptr};
    const lattice *xsrc[2] = {nullptr, nullptr};
    uint64_t xsrc_gen[2] = {0, 0};
    uint64_t xown_gen[2] = {0, 0};
    uint64_t gen = 0;           // incremented by every splat
    // Distribute + PointNet scratch (distribute.hip), allocated on first use.
    int32_t *lvert = nullptr;   // [(d+1) max_points] vertex of each pair-list entry
    double *macc = nullptr;     // [max_vertices][d] position sums of lists that cross a 64-entry chunk
    float *mu = nullptr;        // [max_vertices][d] local means when the caller does not take them
    float *pn_params = nullptr; // the PointNet parameters in the kernel's padded layout
    unsigned int *pn_keys = nullptr;  // [(d+1) max_points / 64 + 1][64] running-max keys of lists
                                      // that cross a 64-entry chunk (row j: the list starting in chunk j)
    // Group normalisation: per cloud, the fp64 sums of each block's input
    // (in copies) and the affines applied.
    double *pn_stats = nullptr;
    float *pn_aff = nullptr;
    int32_t *idx = nullptr;     // [max_points][d+1] hash slot, then vertex index
    int32_t *rank = nullptr;    // [max_points][d+1] position of the pair in its vertex's list
    float *bary = nullptr;      // [max_points][d+1]
    int32_t *list = nullptr;    // [(d+1) max_points][2] (point, weight bits) grouped by vertex
    int32_t *nbr = nullptr;     // [max_vertices][T]
    int32_t *counters = nullptr;  // [CNT_WORDS] device
    uint16_t *zero_row = nullptr; // [512] zeros: the row a missing neighbour reads
    int32_t *host_counters = nullptr;  // pinned [CNT_WORDS]

    int64_t m = 0;
    bool splatted = false;
    bool nbr_valid = false;
    bool batched = false;
    int cu_count = 256;

    int conv_path = LATTICE_CONV_AUTO;  // lattice_set_conv_path

    int timing = 0;
    lattice_timer timers[LATTICE_NUM_STAGES];
    void *events = nullptr;  // per-stage event pools and pending pairs (lattice.hip)
    // With timing on, the events that a stage made of one kernel (slice,
    // deform slice) has its launch record at the kernel's start and end
    // (hipExtLaunchKernelGGL); null otherwise
    hipEvent_t kt_start = nullptr, kt_stop = nullptr;

    char err[512] = {0};
};

// ---- kernel launchers (each returns the launch status) ----

// splat.hip
hipError_t launch_clear_table(lattice *L);
hipError_t launch_insert(lattice *L, const float *pos, const int32_t *batch, int64_t m);
hipError_t launch_number(lattice *L, int64_t m);
hipError_t launch_fill(lattice *L, int64_t m);
hipError_t launch_gather(lattice *L, const float *feat, int C, int normalize, void *values, lattice_dtype values_dt,
                         float *weight);
int64_t split_rows_max(const lattice *L);
int64_t scan_blocks_max();
hipError_t launch_export_keys(lattice *L, int32_t *keys, int32_t *batch);
hipError_t launch_to_bf16(lattice *L, const float *src, int64_t n, uint16_t *dst);

// neighbors.hip
hipError_t launch_neighbors(lattice *L);
hipError_t launch_cross(lattice *out, const lattice *src, bool up, int32_t *xnbr);

// conv.hip
hipError_t launch_conv(lattice *L, const void *in, lattice_dtype in_dt, int C_in, const void *w, int C_out,
                       lattice_dtype dt, const float *bias, void *out, lattice_dtype out_dt);

// slice.hip
hipError_t launch_slice(lattice *L, const void *values, lattice_dtype values_dt, int C, float *out);
hipError_t launch_splat_backward(lattice *L, const void *grad_values, lattice_dtype gv_dt, int C,
                                 const float *vweight, float *grad_feat);

// backward.hip
int wgrad_chunks(const lattice *L, int C_in, int C_out);
hipError_t launch_conv_wgrad(lattice *L, const void *g, lattice_dtype g_dt, int C_out, const void *x,
                             lattice_dtype x_dt, int C_in, lattice_dtype dt, int nch, float *partial,
                             float *pbias, float *grad_w, float *grad_bias);
hipError_t launch_flip_weights(lattice *L, const void *w, bool bf16, int C_out, int C_in, void *wt);

// distribute.hip
hipError_t launch_distribute_pointnet(lattice *L, const float *pos, const float *feat, int f_d, const float *params,
                                      const int *groups, float eps, void *out, bool out_bf16, float *mean);
int64_t pointnet_stats_bytes();
int64_t pointnet_aff_bytes();
int pointnet_param_count(int k0);
int pointnet_padded_count();
int64_t pointnet_backward_scratch_bytes(const lattice *L);
hipError_t launch_distribute_backward(lattice *L, const float *pos, const float *feat, int f_d, const float *params,
                                      const int *groups, float eps, const float *grad_out, float *grad_params,
                                      void *scratch);

// deform.hip
int deform_max_channels(const void *values, lattice_dtype values_dt, int C, const float *w_delta, const float *w_cls,
                        const float *out);
hipError_t launch_deform_slice(lattice *L, const void *values, lattice_dtype values_dt, int C, const float *w_delta,
                               float b_delta, const float *w_cls, const float *b_cls, int n_cls, float *out,
                               float *delta);

// deform_bwd.hip
int64_t deform_backward_scratch_bytes(const lattice *L, int C, int n_cls);
hipError_t launch_deform_backward(lattice *L, const void *values, lattice_dtype values_dt, int C,
                                  const float *w_delta, float b_delta, const float *w_cls, int n_cls,
                                  const float *grad_out, void *grad_values, lattice_dtype grad_dt,
                                  float *grad_w_delta, float *grad_b_delta, float *grad_w_cls, float *grad_b_cls,
                                  void *scratch);

// Workgroups are handed to the eight XCDs round robin (workgroup b runs on
// XCD b % 8, checked on the device), and each XCD has its own L2.  Kernels
// that give each workgroup one contiguous chunk of the work take chunk
// xcd_order(b): the workgroups of one XCD then cover consecutive chunks, so
// that neighbouring items (and the rows they share) meet in the same L2.
// (Measured: this helps the pair-list fill.)
__device__ __forceinline__ int64_t xcd_order(int64_t b, int64_t nb) {
    if (nb % 8 != 0) return b;
    return (b % 8) * (nb / 8) + b / 8;
}

// A grid-stride loop over n items split among the XCDs: XCD x (the one
// workgroup b runs on, b % 8) takes the contiguous range [x n / 8,
// (x + 1) n / 8), and its wavefronts interleave within that range, so that
// items next to each other (and the rows they share) meet in one XCD's L2.
// Without a multiple of 8 workgroups, one range and every wavefront.
struct XcdShare {
    int64_t lo, hi;      // this XCD's items
    int64_t wave, nwaves;  // this wavefront's index among the XCD's, and their number
};
__device__ __forceinline__ XcdShare xcd_share(int64_t n) {
    const int64_t nb = gridDim.x;
    const int64_t wpb = blockDim.x >> 6;
    const int64_t w = threadIdx.x >> 6;
    if (nb % 8 != 0) return {0, n, (int64_t)blockIdx.x * wpb + w, nb * wpb};
    const int64_t x = blockIdx.x % 8;
    return {n * x / 8, n * (x + 1) / 8, (int64_t)(blockIdx.x / 8) * wpb + w, (nb / 8) * wpb};
}

// This workgroup's chunk [lo, hi) of n items, chunks a multiple of `align`.
__device__ __forceinline__ void block_chunk(int64_t n, int64_t align, int64_t &lo, int64_t &hi) {
    const int64_t nb = gridDim.x;
    int64_t per = (n + nb - 1) / nb;
    per = (per + align - 1) / align * align;
    lo = xcd_order(blockIdx.x, nb) * per;
    if (lo > n) lo = n;
    hi = lo + per < n ? lo + per : n;
}

// Grid size for a grid-stride kernel over `work` items with `per_block`
// items per block, capped so that the launch stays a few waves deep.
static inline unsigned grid_for(int64_t work, int64_t per_block, int cu_count, int blocks_per_cu = 8) {
    int64_t g = (work + per_block - 1) / per_block;
    int64_t cap = (int64_t)cu_count * blocks_per_cu;
    if (g > cap) g = cap;
    if (g < 1) g = 1;
    return (unsigned)g;
}
