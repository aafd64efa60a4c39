// Host side of the C ABI declared in include/lattice.h: argument checking,
// ownership of the lattice's device buffers, call ordering, device status,
// and per-stage event timing.  Every kernel is enqueued on the lattice's
// stream; nothing here computes any part of the method on the host except
// the fp32 elevation factors (computed once per lattice in fp64).
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <mutex>
#include <vector>

#include "internal.h"

namespace {

// Workspace of lattice_conv_backward_noalloc: a fixed device array, one copy
// per GPU, held from when the library is loaded on that GPU until the process
// ends.  Host code never uses the name `scratch` as an address (it is a
// host-side stand-in): lattice_create resolves the device address once per
// GPU, with that GPU current, and every use goes through that address.
static __device__ __align__(256) unsigned char scratch[LATTICE_NOALLOC_WORKSPACE_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices] = {};
bool g_scratch_done[kMaxDevices] = {};

// Resolve this GPU's copy of the workspace (the current device must be
// `device`); once per device.
void noalloc_setup(int device) {
    if (device < 0 || device >= kMaxDevices) return;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (g_scratch_done[device]) return;
    g_scratch_done[device] = true;
    void *p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) == hipSuccess)
        g_scratch_ptr[device] = p;
    else
        (void)hipGetLastError();
}

void *noalloc_workspace(int device) {
    if (device < 0 || device >= kMaxDevices) return nullptr;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    return g_scratch_ptr[device];
}

void set_err(lattice *L, const char *fmt, ...) {
    if (!L) return;
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(L->err, sizeof(L->err), fmt, ap);
    va_end(ap);
}

lattice_status hip_fail(lattice *L, hipError_t e, const char *what) {
    set_err(L, "%s: %s", what, hipGetErrorString(e));
    return LATTICE_E_HIP;
}

#define HIP_TRY(L, expr)                                  \
    do {                                                  \
        hipError_t e_ = (expr);                           \
        if (e_ != hipSuccess) return hip_fail(L, e_, #expr); \
    } while (0)

int64_t next_pow2(int64_t x) {
    int64_t p = 64;
    while (p < x) p <<= 1;
    return p;
}

void free_all(lattice *L) {
    (void)hipFree(L->tab);
    (void)hipFree(L->occ);
    (void)hipFree(L->vkeys);
    (void)hipFree(L->vslot);
    (void)hipFree(L->dfb);
    (void)hipFree(L->pnb);
    (void)hipFree(L->blk);
    (void)hipFree(L->split);
    (void)hipFree(L->rowmap);
    (void)hipFree(L->partrec);
    (void)hipFree(L->pweight);
    (void)hipFree(L->partial);
    (void)hipFree(L->wflip);
    (void)hipFree(L->wgpart);
    (void)hipFree(L->xtab[0]);
    (void)hipFree(L->xtab[1]);
    (void)hipFree(L->lvert);
    (void)hipFree(L->macc);
    (void)hipFree(L->mu);
    (void)hipFree(L->pn_params);
    (void)hipFree(L->pn_keys);
    (void)hipFree(L->pn_stats);
    (void)hipFree(L->pn_aff);
    (void)hipFree(L->vinfo);
    (void)hipFree(L->idx);
    (void)hipFree(L->rank);
    (void)hipFree(L->bary);
    (void)hipFree(L->list);
    (void)hipFree(L->nbr);
    (void)hipFree(L->counters);
    (void)hipFree(L->zero_row);
    if (L->host_counters) (void)hipHostFree(L->host_counters);
}

// Event pairs of one stage that have been recorded but not yet read.
struct stage_events {
    std::vector<hipEvent_t> pool;
    std::vector<std::pair<hipEvent_t, hipEvent_t>> pending;
};

stage_events *events_of(lattice *L) { return reinterpret_cast<stage_events *>(L->events); }

lattice_status timer_begin(lattice *L, int stage, hipEvent_t *out) {
    *out = nullptr;
    if (!L->timing) return LATTICE_OK;
    stage_events *se = events_of(L) + stage;
    hipEvent_t e;
    if (!se->pool.empty()) {
        e = se->pool.back();
        se->pool.pop_back();
    } else {
        HIP_TRY(L, hipEventCreate(&e));
    }
    HIP_TRY(L, hipEventRecord(e, L->stream));
    *out = e;
    return LATTICE_OK;
}

lattice_status timer_end(lattice *L, int stage, hipEvent_t start) {
    if (!L->timing || !start) return LATTICE_OK;
    stage_events *se = events_of(L) + stage;
    hipEvent_t e;
    if (!se->pool.empty()) {
        e = se->pool.back();
        se->pool.pop_back();
    } else {
        HIP_TRY(L, hipEventCreate(&e));
    }
    HIP_TRY(L, hipEventRecord(e, L->stream));
    se->pending.emplace_back(start, e);
    return LATTICE_OK;
}

// A stage made of one kernel: two events that its launch records at the
// kernel's start and end (L->kt_start, L->kt_stop), so that the stage's time
// is the kernel's own duration; timer_kernel_end files the pair and clears
// the fields (also after a failed launch).
static lattice_status pool_event(lattice *L, stage_events *se, hipEvent_t *e) {
    if (!se->pool.empty()) {
        *e = se->pool.back();
        se->pool.pop_back();
        return LATTICE_OK;
    }
    HIP_TRY(L, hipEventCreate(e));
    return LATTICE_OK;
}

lattice_status timer_kernel_begin(lattice *L, int stage) {
    L->kt_start = L->kt_stop = nullptr;
    if (!L->timing) return LATTICE_OK;
    stage_events *se = events_of(L) + stage;
    hipEvent_t a, b;
    lattice_status s = pool_event(L, se, &a);
    if (s) return s;
    if ((s = pool_event(L, se, &b))) {
        se->pool.push_back(a);
        return s;
    }
    L->kt_start = a;
    L->kt_stop = b;
    return LATTICE_OK;
}

void timer_kernel_end(lattice *L, int stage, bool launched) {
    if (L->kt_start) {
        stage_events *se = events_of(L) + stage;
        if (launched) {
            se->pending.emplace_back(L->kt_start, L->kt_stop);
        } else {
            se->pool.push_back(L->kt_start);
            se->pool.push_back(L->kt_stop);
        }
    }
    L->kt_start = L->kt_stop = nullptr;
}

lattice_status check_launch(lattice *L, hipError_t e, const char *what) {
    if (e != hipSuccess) return hip_fail(L, e, what);
    return LATTICE_OK;
}

// Copy the first V rows (V on the device) of an int32 or fp32 table.
__global__ void k_copy_rows(const uint32_t *__restrict__ src, uint32_t *__restrict__ dst, int64_t row_words,
                            const int32_t *counters, int64_t fixed_rows) {
    const int64_t rows = fixed_rows >= 0 ? fixed_rows : (int64_t)counters[CNT_V];
    const int64_t n = rows * row_words;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) dst[i] = src[i];
}

lattice_status copy_rows(lattice *L, const void *src, void *dst, int64_t row_words, int64_t fixed_rows,
                         int64_t bound_rows) {
    const unsigned grid = grid_for(bound_rows * row_words, 256, L->cu_count, 4);
    hipLaunchKernelGGL(k_copy_rows, dim3(grid), dim3(256), 0, L->stream, reinterpret_cast<const uint32_t *>(src),
                       reinterpret_cast<uint32_t *>(dst), row_words, L->counters, fixed_rows);
    return check_launch(L, hipGetLastError(), "copy_rows");
}

// Grow a scratch buffer of the lattice to at least `need` bytes (a device
// allocation, only when it is too small).
lattice_status grow(lattice *L, void **buf, int64_t *have, int64_t need, const char *what) {
    if (need <= *have) return LATTICE_OK;
    if (*buf) HIP_TRY(L, hipFree(*buf));
    *buf = nullptr;
    *have = 0;
    if (hipMalloc(buf, need) != hipSuccess) {
        (void)hipGetLastError();
        *buf = nullptr;
        set_err(L, "%s: cannot allocate %lld bytes of scratch", what, (long long)need);
        return LATTICE_E_NOMEM;
    }
    *have = need;
    return LATTICE_OK;
}

// The gather scratch (partial rows of long pair lists) sized for C columns.
lattice_status ensure_partial(lattice *L, int C, const char *what) {
    const int64_t cols = (C + 3) & ~3;
    if (cols <= L->partial_cols) return LATTICE_OK;
    int64_t have = L->partial_cols * split_rows_max(L) * (int64_t)sizeof(float);
    void *buf = L->partial;
    lattice_status s = grow(L, &buf, &have, split_rows_max(L) * cols * (int64_t)sizeof(float), what);
    L->partial = reinterpret_cast<float *>(buf);
    L->partial_cols = s == LATTICE_OK ? cols : 0;
    return s;
}

lattice_status ensure_neighbors(lattice *L) {
    if (L->nbr_valid) return LATTICE_OK;
    hipEvent_t t0;
    lattice_status s = timer_begin(L, LATTICE_STAGE_NEIGHBORS, &t0);
    if (s) return s;
    s = check_launch(L, launch_neighbors(L), "neighbors");
    if (s) return s;
    s = timer_end(L, LATTICE_STAGE_NEIGHBORS, t0);
    if (s) return s;
    L->nbr_valid = true;
    return LATTICE_OK;
}

}  // namespace

extern "C" {

const char *lattice_status_string(lattice_status s) {
    switch (s) {
        case LATTICE_OK: return "ok";
        case LATTICE_E_ARG: return "invalid argument";
        case LATTICE_E_STATE: return "call out of order";
        case LATTICE_E_RANGE: return "key coordinate or batch id out of range";
        case LATTICE_E_CAPACITY: return "hash table full";
        case LATTICE_E_NOMEM: return "out of memory";
        case LATTICE_E_HIP: return "HIP runtime error";
    }
    return "unknown status";
}

const char *lattice_last_error(const lattice *L) { return L ? L->err : "null lattice"; }

lattice_status lattice_create(int d, const float *sigma, double alpha, int64_t max_points, int64_t hash_capacity,
                              void *stream, lattice **out) {
    if (!out) return LATTICE_E_ARG;
    *out = nullptr;
    if (d < 1 || d > LATTICE_MAX_D || !sigma || max_points < 1 || max_points > (int64_t)1 << 28 ||
        hash_capacity < 0 || hash_capacity > (int64_t)1 << 30)
        return LATTICE_E_ARG;
    for (int j = 0; j < d; ++j)
        if (!(sigma[j] > 0.f) || !isfinite(sigma[j])) return LATTICE_E_ARG;
    if (!isfinite(alpha)) return LATTICE_E_ARG;

    lattice *L = new (std::nothrow) lattice();
    if (!L) return LATTICE_E_NOMEM;
    L->d = d;
    L->T = LATTICE_TAPS(d);
    L->alpha = alpha > 0 ? alpha : (d + 1) * sqrt(2.0 / 3.0);
    for (int j = 1; j <= d; ++j) {
        L->sigma[j - 1] = sigma[j - 1];
        L->factors[j - 1] = (float)(L->alpha / ((double)sigma[j - 1] * sqrt((double)(j * (j + 1)))));
    }
    L->inv_dp1 = (float)(1.0 / (d + 1));
    L->max_points = max_points;
    const int64_t keys_max = (int64_t)(d + 1) * max_points;
    // default: room for every pair's vertex with a third of the slots to
    // spare, so that the linear probe chains of lookups that fail (most ring
    // neighbours of a sparse scan are absent) stay short at the worst load
    L->cap = next_pow2(hash_capacity > 0 ? hash_capacity : (3 * keys_max + 1) / 2);
    if (L->cap > (int64_t)1 << 30) {
        delete L;
        return LATTICE_E_ARG;
    }
    L->max_vertices = keys_max < L->cap ? keys_max : L->cap;
    L->stream = reinterpret_cast<hipStream_t>(stream);

    hipError_t e = hipGetDevice(&L->device);
    if (e != hipSuccess) {
        delete L;
        return LATTICE_E_HIP;
    }
    int cus = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, L->device) == hipSuccess && cus > 0)
        L->cu_count = cus;
    noalloc_setup(L->device);

    const int dp1 = d + 1;
    bool ok = hipMalloc(&L->tab, L->cap * 16) == hipSuccess &&
              hipMalloc(&L->occ, (size_t)(L->cap + 31) / 32 * 4) == hipSuccess &&
              hipMalloc(&L->vkeys, L->max_vertices * sizeof(uint64_t)) == hipSuccess &&
              hipMalloc(&L->vslot, L->max_vertices * sizeof(int32_t)) == hipSuccess &&
              hipMalloc(&L->blk, scan_blocks_max() * 4 * sizeof(int32_t)) == hipSuccess &&
              hipMalloc(&L->split, split_rows_max(L) * 3 * sizeof(int32_t)) == hipSuccess &&
              hipMalloc(&L->rowmap, split_rows_max(L) * sizeof(int32_t)) == hipSuccess &&
              hipMalloc(&L->partrec, split_rows_max(L) * 2 * sizeof(int32_t)) == hipSuccess &&
              hipMalloc(&L->pweight, split_rows_max(L) * sizeof(float)) == hipSuccess &&
              hipMalloc(&L->vinfo, L->max_vertices * 2 * sizeof(int32_t)) == hipSuccess &&
              hipMalloc(&L->idx, max_points * dp1 * sizeof(int32_t)) == hipSuccess &&
              hipMalloc(&L->rank, max_points * dp1 * sizeof(int32_t)) == hipSuccess &&
              hipMalloc(&L->bary, max_points * dp1 * sizeof(float)) == hipSuccess &&
              hipMalloc(&L->list, max_points * dp1 * 2 * sizeof(int32_t)) == hipSuccess &&
              hipMalloc(&L->nbr, L->max_vertices * L->T * sizeof(int32_t)) == hipSuccess &&
              hipMalloc(&L->counters, CNT_WORDS * sizeof(int32_t)) == hipSuccess &&
              hipMalloc(&L->zero_row, 512 * sizeof(uint16_t)) == hipSuccess &&
              hipMemset(L->zero_row, 0, 512 * sizeof(uint16_t)) == hipSuccess &&
              hipHostMalloc(&L->host_counters, CNT_WORDS * sizeof(int32_t), hipHostMallocDefault) == hipSuccess;
    if (!ok) {
        (void)hipGetLastError();
        free_all(L);
        delete L;
        return LATTICE_E_NOMEM;
    }
    L->events = new (std::nothrow) stage_events[LATTICE_NUM_STAGES];
    if (!L->events) {
        free_all(L);
        delete L;
        return LATTICE_E_NOMEM;
    }
    *out = L;
    return LATTICE_OK;
}

void lattice_destroy(lattice *L) {
    if (!L) return;
    (void)hipStreamSynchronize(L->stream);
    stage_events *se = events_of(L);
    if (se) {
        for (int s = 0; s < LATTICE_NUM_STAGES; ++s) {
            for (auto &pr : se[s].pending) {
                (void)hipEventDestroy(pr.first);
                (void)hipEventDestroy(pr.second);
            }
            for (auto e : se[s].pool) (void)hipEventDestroy(e);
        }
        delete[] se;
    }
    free_all(L);
    delete L;
}

int64_t lattice_max_vertices(const lattice *L, int64_t m) {
    if (!L || m < 0) return -1;
    const int64_t k = (int64_t)(L->d + 1) * m;
    return k < L->cap ? k : L->cap;
}

int64_t lattice_hash_capacity(const lattice *L) { return L ? L->cap : -1; }
int lattice_dim(const lattice *L) { return L ? L->d : -1; }

lattice_status lattice_splat(lattice *L, const float *pos, const int32_t *batch, int64_t m, const float *feat, int C,
                             int normalize, void *values, lattice_dtype values_dtype, float *weight) {
    if (!L) return LATTICE_E_ARG;
    if (m < 0 || m > L->max_points) {
        set_err(L, "splat: m = %lld outside [0, %lld]", (long long)m, (long long)L->max_points);
        return LATTICE_E_ARG;
    }
    if (C < 0 || C > 4096 || (m > 0 && !pos) || (m > 0 && C > 0 && !feat) || (m > 0 && C > 0 && !values) ||
        (values_dtype != LATTICE_F32 && values_dtype != LATTICE_BF16)) {
        set_err(L, "splat: bad pointer or channel count (C = %d)", C);
        return LATTICE_E_ARG;
    }
    if (batch && L->d == 4) {
        set_err(L, "splat: batch ids need d <= 3 (a d = 4 key uses all 64 bits)");
        return LATTICE_E_ARG;
    }
    // Scratch for the partial rows of long pair lists, sized for C columns
    // (grown here, outside any timed or captured region of a caller that
    // splats once before it times or captures).
    lattice_status s = ensure_partial(L, C, "splat");
    if (s) return s;
    hipEvent_t t0;
    if ((s = timer_begin(L, LATTICE_STAGE_SPLAT, &t0))) return s;
    // The slots to empty are those the last splat listed; until this splat's
    // launches have all gone out, the next one empties the whole table.
    if ((s = check_launch(L, launch_clear_table(L), "clear_table"))) return s;
    L->full_clear = true;
    if ((s = check_launch(L, launch_insert(L, pos, batch, m), "insert"))) return s;
    if ((s = check_launch(L, launch_number(L, m), "number"))) return s;
    if ((s = check_launch(L, launch_fill(L, m), "fill"))) return s;
    if (C > 0 || weight)
        if ((s = check_launch(L, launch_gather(L, feat, C, normalize, values, values_dtype, weight), "gather")))
            return s;
    if ((s = timer_end(L, LATTICE_STAGE_SPLAT, t0))) return s;
    L->full_clear = false;
    L->m = m;
    L->gen += 1;
    L->splatted = true;
    L->nbr_valid = false;
    L->batched = batch != nullptr;
    return LATTICE_OK;
}

lattice_status lattice_set_conv_path(lattice *L, int path) {
    if (!L) return LATTICE_E_ARG;
    if (path < LATTICE_CONV_AUTO || path > LATTICE_CONV_RS) {
        set_err(L, "set_conv_path: unknown path %d", path);
        return LATTICE_E_ARG;
    }
    L->conv_path = path;
    return LATTICE_OK;
}

lattice_status lattice_build_neighbors(lattice *L) {
    if (!L) return LATTICE_E_ARG;
    if (!L->splatted) {
        set_err(L, "build_neighbors: no lattice yet (call lattice_splat first)");
        return LATTICE_E_STATE;
    }
    return ensure_neighbors(L);
}

lattice_status lattice_conv(lattice *L, const void *in, lattice_dtype in_dtype, int C_in, const void *w, int C_out,
                            lattice_dtype dt, const float *bias, void *out, lattice_dtype out_dtype) {
    if (!L) return LATTICE_E_ARG;
    if (!L->splatted) {
        set_err(L, "conv: no lattice yet (call lattice_splat first)");
        return LATTICE_E_STATE;
    }
    if (!in || !w || !out || C_in < 1 || C_in > 1024 || C_out < 1 || C_out > 1024 ||
        (dt != LATTICE_F32 && dt != LATTICE_BF16) || (in_dtype != LATTICE_F32 && in_dtype != LATTICE_BF16) ||
        (out_dtype != LATTICE_F32 && out_dtype != LATTICE_BF16) || in == out) {
        set_err(L, "conv: bad argument (C_in = %d, C_out = %d, dtype = %d)", C_in, C_out, (int)dt);
        return LATTICE_E_ARG;
    }
    lattice_status s = ensure_neighbors(L);
    if (s) return s;
    hipEvent_t t0;
    if ((s = timer_begin(L, LATTICE_STAGE_CONV, &t0))) return s;
    if ((s = check_launch(L, launch_conv(L, in, in_dtype, C_in, w, C_out, dt, bias, out, out_dtype), "conv")))
        return s;
    return timer_end(L, LATTICE_STAGE_CONV, t0);
}

lattice_status lattice_slice(lattice *L, const void *values, lattice_dtype values_dtype, int C, float *out) {
    if (!L) return LATTICE_E_ARG;
    if (!L->splatted) {
        set_err(L, "slice: no lattice yet (call lattice_splat first)");
        return LATTICE_E_STATE;
    }
    if (C < 1 || C > 4096 || (L->m > 0 && (!values || !out)) ||
        (values_dtype != LATTICE_F32 && values_dtype != LATTICE_BF16)) {
        set_err(L, "slice: bad argument (C = %d)", C);
        return LATTICE_E_ARG;
    }
    lattice_status s = timer_kernel_begin(L, LATTICE_STAGE_SLICE);
    if (s) return s;
    const hipError_t e = launch_slice(L, values, values_dtype, C, out);
    timer_kernel_end(L, LATTICE_STAGE_SLICE, e == hipSuccess && L->m > 0);
    return check_launch(L, e, "slice");
}

lattice_status lattice_deform_slice(lattice *L, const void *values, lattice_dtype values_dtype, int C,
                                    const float *w_delta, float b_delta, const float *w_cls, const float *b_cls,
                                    int n_cls, float *out, float *delta) {
    if (!L) return LATTICE_E_ARG;
    if (!L->splatted) {
        set_err(L, "deform_slice: no lattice yet (call lattice_splat first)");
        return LATTICE_E_STATE;
    }
    if (C < 1 || (values_dtype != LATTICE_F32 && values_dtype != LATTICE_BF16) || (w_cls && (n_cls < 1 || n_cls > 256)) ||
        (!w_cls && b_cls) || (L->m > 0 && (!values || !w_delta || !out))) {
        set_err(L, "deform_slice: bad argument (C = %d, n_cls = %d)", C, n_cls);
        return LATTICE_E_ARG;
    }
    const int cmax = deform_max_channels(values, values_dtype, C, w_delta, w_cls, out);
    if (C > cmax) {
        set_err(L, "deform_slice: C = %d above %d (C above 256 needs a multiple of 4 and aligned rows)", C, cmax);
        return LATTICE_E_ARG;
    }
    lattice_status s = timer_kernel_begin(L, LATTICE_STAGE_DEFORM);
    if (s) return s;
    const hipError_t e =
        launch_deform_slice(L, values, values_dtype, C, w_delta, b_delta, w_cls, b_cls, n_cls, out, delta);
    timer_kernel_end(L, LATTICE_STAGE_DEFORM, e == hipSuccess && L->m > 0);
    return check_launch(L, e, "deform_slice");
}

lattice_status lattice_deform_slice_backward(lattice *L, const void *values, lattice_dtype values_dtype, int C,
                                             const float *w_delta, float b_delta, const float *w_cls, int n_cls,
                                             const float *grad_out, void *grad_values, lattice_dtype grad_dtype,
                                             float *grad_w_delta, float *grad_b_delta, float *grad_w_cls,
                                             float *grad_b_cls) {
    if (!L) return LATTICE_E_ARG;
    if (!L->splatted) {
        set_err(L, "deform_slice_backward: no lattice yet (call lattice_splat first)");
        return LATTICE_E_STATE;
    }
    auto bad_dt = [](lattice_dtype t) { return t != LATTICE_F32 && t != LATTICE_BF16; };
    const bool any_out = grad_values || grad_w_delta || grad_b_delta || grad_w_cls || grad_b_cls;
    if (C < 1 || C > 1024 || bad_dt(values_dtype) || bad_dt(grad_dtype) || (w_cls && (n_cls < 1 || n_cls > 256)) ||
        (!w_cls && (grad_w_cls || grad_b_cls)) || !any_out || (L->m > 0 && (!values || !grad_out)) || !w_delta ||
        (grad_values && (grad_values == values || grad_values == (const void *)grad_out))) {
        set_err(L, "deform_slice_backward: bad argument (C = %d, n_cls = %d)", C, n_cls);
        return LATTICE_E_ARG;
    }
    const int ncls = w_cls ? n_cls : 0;
    lattice_status s = grow(L, &L->dfb, &L->dfb_bytes, deform_backward_scratch_bytes(L, C, ncls),
                            "deform_slice_backward");
    if (s) return s;
    hipEvent_t t0;
    if ((s = timer_begin(L, LATTICE_STAGE_DEFORM_BACKWARD, &t0))) return s;
    if ((s = check_launch(L,
                          launch_deform_backward(L, values, values_dtype, C, w_delta, b_delta, w_cls, ncls, grad_out,
                                                 grad_values, grad_dtype, grad_w_delta, grad_b_delta, grad_w_cls,
                                                 grad_b_cls, L->dfb),
                          "deform_slice_backward")))
        return s;
    return timer_end(L, LATTICE_STAGE_DEFORM_BACKWARD, t0);
}

lattice_status lattice_slice_backward(lattice *L, const float *grad_out, int C, void *grad_values,
                                      lattice_dtype grad_dtype) {
    if (!L) return LATTICE_E_ARG;
    if (!L->splatted) {
        set_err(L, "slice_backward: no lattice yet (call lattice_splat first)");
        return LATTICE_E_STATE;
    }
    if (C < 1 || C > 4096 || (L->m > 0 && (!grad_out || !grad_values)) ||
        (grad_dtype != LATTICE_F32 && grad_dtype != LATTICE_BF16) ||
        (grad_values && (const void *)grad_out == grad_values)) {
        set_err(L, "slice_backward: bad argument (C = %d)", C);
        return LATTICE_E_ARG;
    }
    lattice_status s = ensure_partial(L, C, "slice_backward");
    if (s) return s;
    hipEvent_t t0;
    if ((s = timer_begin(L, LATTICE_STAGE_SLICE_BACKWARD, &t0))) return s;
    // Eq. (splat) of the point gradients over the pair lists of the last splat
    if ((s = check_launch(L, launch_gather(L, grad_out, C, 0, grad_values, grad_dtype, nullptr), "slice_backward")))
        return s;
    return timer_end(L, LATTICE_STAGE_SLICE_BACKWARD, t0);
}

lattice_status lattice_splat_backward(lattice *L, const void *grad_values, lattice_dtype gv_dtype, int C,
                                      int normalize, const float *weight, float *grad_feat) {
    if (!L) return LATTICE_E_ARG;
    if (!L->splatted) {
        set_err(L, "splat_backward: no lattice yet (call lattice_splat first)");
        return LATTICE_E_STATE;
    }
    if (C < 1 || C > 4096 || (normalize != 0 && normalize != 1) || (normalize && !weight) ||
        (L->m > 0 && (!grad_values || !grad_feat)) || (gv_dtype != LATTICE_F32 && gv_dtype != LATTICE_BF16)) {
        set_err(L, "splat_backward: bad argument (C = %d, normalize = %d)", C, normalize);
        return LATTICE_E_ARG;
    }
    hipEvent_t t0;
    lattice_status s = timer_begin(L, LATTICE_STAGE_SPLAT_BACKWARD, &t0);
    if (s) return s;
    // Eq. (slice) of the vertex gradients (divided by w_v for the normalised splat)
    if ((s = check_launch(L, launch_splat_backward(L, grad_values, gv_dtype, C, normalize ? weight : nullptr,
                                                   grad_feat),
                          "splat_backward")))
        return s;
    return timer_end(L, LATTICE_STAGE_SPLAT_BACKWARD, t0);
}

// Argument checks shared by the two conv backward entry points.
static lattice_status conv_backward_args(lattice *L, const void *grad_out, lattice_dtype g_dtype, int C_out,
                                         const void *w, int C_in, lattice_dtype dt, const void *in,
                                         lattice_dtype in_dtype, void *grad_in, lattice_dtype grad_in_dtype,
                                         float *grad_w, float *grad_bias, const char *what) {
    if (!L) return LATTICE_E_ARG;
    if (!L->splatted) {
        set_err(L, "%s: no lattice yet (call lattice_splat first)", what);
        return LATTICE_E_STATE;
    }
    auto bad_dt = [](lattice_dtype t) { return t != LATTICE_F32 && t != LATTICE_BF16; };
    if (!grad_out || C_out < 1 || C_out > 1024 || C_in < 1 || C_in > 1024 || bad_dt(g_dtype) || bad_dt(dt) ||
        (grad_in && (!w || bad_dt(grad_in_dtype) || grad_in == grad_out)) ||
        ((grad_w || grad_bias) && !in) || (in && bad_dt(in_dtype)) || (!grad_in && !grad_w && !grad_bias)) {
        set_err(L, "%s: bad argument (C_out = %d, C_in = %d)", what, C_out, C_in);
        return LATTICE_E_ARG;
    }
    return LATTICE_OK;
}

// The launches of a conv backward, with the flipped weights in `wflip` and
// the weight-gradient partials (then the bias partials) in `wgpart`.
static lattice_status conv_backward_run(lattice *L, const void *grad_out, lattice_dtype g_dtype, int C_out,
                                        const void *w, int C_in, lattice_dtype dt, const void *in,
                                        lattice_dtype in_dtype, void *grad_in, lattice_dtype grad_in_dtype,
                                        float *grad_w, float *grad_bias, int nch, void *wflip, float *wgpart) {
    lattice_status s;
    if (grad_in) {
        // dx = forward conv of g with W'[i][s][o] = W[o][flip(s)][i]
        if ((s = check_launch(L, launch_flip_weights(L, w, dt == LATTICE_BF16, C_out, C_in, wflip),
                              "conv_backward flip")))
            return s;
        if ((s = check_launch(L, launch_conv(L, grad_out, g_dtype, C_out, wflip, C_in, dt, nullptr, grad_in,
                                             grad_in_dtype),
                              "conv_backward input")))
            return s;
    }
    if (grad_w || grad_bias) {
        float *pbias = wgpart + (int64_t)nch * C_out * L->T * C_in;
        if ((s = check_launch(L, launch_conv_wgrad(L, grad_out, g_dtype, C_out, in, in_dtype, C_in, dt, nch, wgpart,
                                                   pbias, grad_w, grad_bias),
                              "conv_backward weight")))
            return s;
    }
    return LATTICE_OK;
}

lattice_status lattice_conv_backward(lattice *L, const void *grad_out, lattice_dtype g_dtype, int C_out,
                                     const void *w, int C_in, lattice_dtype dt, const void *in,
                                     lattice_dtype in_dtype, void *grad_in, lattice_dtype grad_in_dtype,
                                     float *grad_w, float *grad_bias) {
    lattice_status s = conv_backward_args(L, grad_out, g_dtype, C_out, w, C_in, dt, in, in_dtype, grad_in,
                                          grad_in_dtype, grad_w, grad_bias, "conv_backward");
    if (s) return s;
    if ((s = ensure_neighbors(L))) return s;
    const int T = L->T;
    const int nch = wgrad_chunks(L, C_in, C_out);
    if (grad_in) {
        const int64_t esz = dt == LATTICE_BF16 ? 2 : 4;
        if ((s = grow(L, &L->wflip, &L->wflip_bytes, (int64_t)C_out * T * C_in * esz, "conv_backward"))) return s;
    }
    if (grad_w || grad_bias) {
        void *buf = L->wgpart;
        int64_t have = L->wgpart_floats * (int64_t)sizeof(float);
        const int64_t need = (int64_t)nch * ((int64_t)C_out * T * C_in + C_out) * (int64_t)sizeof(float);
        s = grow(L, &buf, &have, need, "conv_backward");
        L->wgpart = reinterpret_cast<float *>(buf);
        L->wgpart_floats = have / (int64_t)sizeof(float);
        if (s) return s;
    }
    hipEvent_t t0;
    if ((s = timer_begin(L, LATTICE_STAGE_CONV_BACKWARD, &t0))) return s;
    if ((s = conv_backward_run(L, grad_out, g_dtype, C_out, w, C_in, dt, in, in_dtype, grad_in, grad_in_dtype, grad_w,
                               grad_bias, nch, L->wflip, L->wgpart)))
        return s;
    return timer_end(L, LATTICE_STAGE_CONV_BACKWARD, t0);
}

lattice_status lattice_conv_backward_noalloc(lattice *L, const void *grad_out, lattice_dtype g_dtype, int C_out,
                                             const void *w, int C_in, lattice_dtype dt, const void *in,
                                             lattice_dtype in_dtype, void *grad_in, lattice_dtype grad_in_dtype,
                                             float *grad_w, float *grad_bias) {
    lattice_status s = conv_backward_args(L, grad_out, g_dtype, C_out, w, C_in, dt, in, in_dtype, grad_in,
                                          grad_in_dtype, grad_w, grad_bias, "conv_backward_noalloc");
    if (s) return s;
    unsigned char *ws = reinterpret_cast<unsigned char *>(noalloc_workspace(L->device));
    if (!ws) {
        set_err(L, "conv_backward_noalloc: the workspace of device %d is not available", L->device);
        return LATTICE_E_HIP;
    }
    const int T = L->T;
    const int nch = wgrad_chunks(L, C_in, C_out);
    // [flipped weights, padded to 256 bytes][partials of the weight and bias gradients]
    const int64_t flip_bytes = grad_in ? ((int64_t)C_out * T * C_in * (dt == LATTICE_BF16 ? 2 : 4) + 255) / 256 * 256 : 0;
    const int64_t part_bytes =
        (grad_w || grad_bias) ? (int64_t)nch * ((int64_t)C_out * T * C_in + C_out) * (int64_t)sizeof(float) : 0;
    if (flip_bytes + part_bytes > (int64_t)LATTICE_NOALLOC_WORKSPACE_BYTES) {
        set_err(L, "conv_backward_noalloc: C_out = %d, C_in = %d, T = %d needs %lld bytes of workspace, above the "
                "%lld available", C_out, C_in, T, (long long)(flip_bytes + part_bytes),
                (long long)LATTICE_NOALLOC_WORKSPACE_BYTES);
        return LATTICE_E_ARG;
    }
    // the neighbour table, without the stage timer (whose events the timer
    // would create on first use)
    if (!L->nbr_valid) {
        if ((s = check_launch(L, launch_neighbors(L), "neighbors"))) return s;
        L->nbr_valid = true;
    }
    // Every element of the workspace that the kernels read is written first
    // in this call (each chunk writes its whole partial tile), so no clearing.
    return conv_backward_run(L, grad_out, g_dtype, C_out, w, C_in, dt, in, in_dtype, grad_in, grad_in_dtype, grad_w,
                             grad_bias, nch, ws, reinterpret_cast<float *>(ws + flip_bytes));
}

// Checks of a lattice pair for down (up = false) or upsampling from `src`
// onto the vertices of `dst`.
static lattice_status resample_pair(lattice *src, lattice *dst, bool up, const char *what) {
    if (!src || !dst) return LATTICE_E_ARG;
    if (!src->splatted || !dst->splatted) {
        set_err(dst, "%s: both lattices must be splatted first", what);
        return LATTICE_E_STATE;
    }
    if (src == dst || src->d != dst->d || src->stream != dst->stream || src->batched != dst->batched ||
        src->device != dst->device) {
        set_err(dst, "%s: the lattices differ in d, stream, device or batching (or are the same)", what);
        return LATTICE_E_ARG;
    }
    // The coarse lattice is the fine one at twice the scale (positions
    // divided by 2), the same alpha.  This also rejects the two lattices
    // passed in the wrong order, whose table would index past the input rows.
    const lattice *fine = up ? dst : src, *coarse = up ? src : dst;
    bool scales = fine->alpha == coarse->alpha;
    for (int j = 0; j < fine->d; ++j) scales = scales && coarse->sigma[j] == 2.f * fine->sigma[j];
    if (!scales) {
        set_err(dst, "%s: the coarse lattice must have exactly twice the fine lattice's sigma and the same alpha "
                "(source and destination in the order of the call)", what);
        return LATTICE_E_ARG;
    }
    return LATTICE_OK;
}

// The table of `dst` (one row of T indices per vertex of dst) into the rows
// of `src`: downsampling 2c' + offset_t, upsampling (u + offset_t) / 2.
// Built on first use and again after either lattice is splatted.
static lattice_status cross_table(lattice *dst, lattice *src, bool up, const char *what, int32_t **table) {
    const int k = up ? 1 : 0;
    if (!dst->xtab[k]) {
        if (hipMalloc(&dst->xtab[k], dst->max_vertices * (int64_t)dst->T * sizeof(int32_t)) != hipSuccess) {
            (void)hipGetLastError();
            dst->xtab[k] = nullptr;
            set_err(dst, "%s: cannot allocate the cross-lattice table", what);
            return LATTICE_E_NOMEM;
        }
        dst->xsrc[k] = nullptr;
    }
    if (dst->xsrc[k] != src || dst->xsrc_gen[k] != src->gen || dst->xown_gen[k] != dst->gen) {
        lattice_status s = check_launch(dst, launch_cross(dst, src, up, dst->xtab[k]), what);
        if (s) return s;
        dst->xsrc[k] = src;
        dst->xsrc_gen[k] = src->gen;
        dst->xown_gen[k] = dst->gen;
    }
    *table = dst->xtab[k];
    return LATTICE_OK;
}

// Down (up = false) or upsampling from `src` onto the vertices of `dst`.
static lattice_status resample(lattice *src, lattice *dst, bool up, const void *in, lattice_dtype in_dtype, int C_in,
                               const void *w, int C_out, lattice_dtype dt, const float *bias, void *out,
                               lattice_dtype out_dtype) {
    const char *what = up ? "upsample" : "downsample";
    lattice_status s = resample_pair(src, dst, up, what);
    if (s) return s;
    if (!in || !w || !out || C_in < 1 || C_in > 1024 || C_out < 1 || C_out > 1024 ||
        (dt != LATTICE_F32 && dt != LATTICE_BF16) || (in_dtype != LATTICE_F32 && in_dtype != LATTICE_BF16) ||
        (out_dtype != LATTICE_F32 && out_dtype != LATTICE_BF16) || in == out) {
        set_err(dst, "%s: bad argument (C_in = %d, C_out = %d)", what, C_in, C_out);
        return LATTICE_E_ARG;
    }
    hipEvent_t t0;
    const int stage = up ? LATTICE_STAGE_UPSAMPLE : LATTICE_STAGE_DOWNSAMPLE;
    if ((s = timer_begin(dst, stage, &t0))) return s;
    int32_t *table = nullptr;
    if ((s = cross_table(dst, src, up, what, &table))) return s;
    // the conv kernels over the output lattice's vertices, reading rows of
    // the source lattice through the cross table
    lattice view = *dst;
    view.nbr = table;
    if ((s = check_launch(dst, launch_conv(&view, in, in_dtype, C_in, w, C_out, dt, bias, out, out_dtype), what)))
        return s;
    return timer_end(dst, stage, t0);
}

// Gradients of resample(src -> dst, up) given grad_out on dst's vertices.
// Both are adjoints that reuse the forward kernels:
//   grad_in (rows of src): the resampling in the other direction (dst -> src)
//     of grad_out with W'[i][s][o] = W[o][flip(s)][i]: downsampling reads
//     fine 2c' + offset_t, so fine u receives from the coarse c' with
//     c' = (u - offset_t) / 2 = (u + offset_flip(t)) / 2, which is tap
//     flip(t) of the upsampling table, and the other way round;
//   grad_w, grad_bias: the conv weight gradient over dst's vertices with the
//     forward's cross table (dW_t = sum over v of g_v^T x_{table(v,t)}).
static lattice_status resample_backward(lattice *src, lattice *dst, bool up, const void *grad_out,
                                        lattice_dtype g_dtype, int C_out, const void *w, int C_in, lattice_dtype dt,
                                        const void *in, lattice_dtype in_dtype, void *grad_in,
                                        lattice_dtype grad_in_dtype, float *grad_w, float *grad_bias) {
    const char *what = up ? "upsample_backward" : "downsample_backward";
    lattice_status s = resample_pair(src, dst, up, what);
    if (s) return s;
    if ((s = conv_backward_args(dst, grad_out, g_dtype, C_out, w, C_in, dt, in, in_dtype, grad_in, grad_in_dtype,
                                grad_w, grad_bias, what)))
        return s;
    if (in && in == grad_in) {
        set_err(dst, "%s: grad_in must not overlap the forward input", what);
        return LATTICE_E_ARG;
    }
    const int T = dst->T;
    const int nch = (grad_w || grad_bias) ? wgrad_chunks(dst, C_in, C_out) : 0;
    if (grad_in) {
        const int64_t esz = dt == LATTICE_BF16 ? 2 : 4;
        if ((s = grow(src, &src->wflip, &src->wflip_bytes, (int64_t)C_out * T * C_in * esz, what))) return s;
    }
    if (grad_w || grad_bias) {
        void *buf = dst->wgpart;
        int64_t have = dst->wgpart_floats * (int64_t)sizeof(float);
        const int64_t need = (int64_t)nch * ((int64_t)C_out * T * C_in + C_out) * (int64_t)sizeof(float);
        s = grow(dst, &buf, &have, need, what);
        dst->wgpart = reinterpret_cast<float *>(buf);
        dst->wgpart_floats = have / (int64_t)sizeof(float);
        if (s) return s;
    }
    hipEvent_t t0;
    const int stage = up ? LATTICE_STAGE_UPSAMPLE_BACKWARD : LATTICE_STAGE_DOWNSAMPLE_BACKWARD;
    if ((s = timer_begin(dst, stage, &t0))) return s;
    if (grad_in) {
        int32_t *back = nullptr;
        if ((s = cross_table(src, dst, !up, what, &back))) return s;
        if ((s = check_launch(src, launch_flip_weights(src, w, dt == LATTICE_BF16, C_out, C_in, src->wflip),
                              what)))
            return s;
        lattice view = *src;
        view.nbr = back;
        if ((s = check_launch(src, launch_conv(&view, grad_out, g_dtype, C_out, src->wflip, C_in, dt, nullptr, grad_in,
                                               grad_in_dtype),
                              what)))
            return s;
    }
    if (grad_w || grad_bias) {
        int32_t *fwd = nullptr;
        if ((s = cross_table(dst, src, up, what, &fwd))) return s;
        lattice view = *dst;
        view.nbr = fwd;
        float *pbias = dst->wgpart + (int64_t)nch * C_out * T * C_in;
        if ((s = check_launch(dst, launch_conv_wgrad(&view, grad_out, g_dtype, C_out, in, in_dtype, C_in, dt, nch,
                                                     dst->wgpart, pbias, grad_w, grad_bias),
                              what)))
            return s;
    }
    return timer_end(dst, stage, t0);
}

lattice_status lattice_downsample(lattice *fine, lattice *coarse, const void *in, lattice_dtype in_dtype, int C_in,
                                  const void *w, int C_out, lattice_dtype dt, const float *bias, void *out,
                                  lattice_dtype out_dtype) {
    return resample(fine, coarse, false, in, in_dtype, C_in, w, C_out, dt, bias, out, out_dtype);
}

lattice_status lattice_upsample(lattice *coarse, lattice *fine, const void *in, lattice_dtype in_dtype, int C_in,
                                const void *w, int C_out, lattice_dtype dt, const float *bias, void *out,
                                lattice_dtype out_dtype) {
    return resample(coarse, fine, true, in, in_dtype, C_in, w, C_out, dt, bias, out, out_dtype);
}

lattice_status lattice_downsample_backward(lattice *fine, lattice *coarse, const void *grad_out,
                                           lattice_dtype g_dtype, int C_out, const void *w, int C_in,
                                           lattice_dtype dt, const void *in, lattice_dtype in_dtype, void *grad_in,
                                           lattice_dtype grad_in_dtype, float *grad_w, float *grad_bias) {
    return resample_backward(fine, coarse, false, grad_out, g_dtype, C_out, w, C_in, dt, in, in_dtype, grad_in,
                             grad_in_dtype, grad_w, grad_bias);
}

lattice_status lattice_upsample_backward(lattice *coarse, lattice *fine, const void *grad_out, lattice_dtype g_dtype,
                                         int C_out, const void *w, int C_in, lattice_dtype dt, const void *in,
                                         lattice_dtype in_dtype, void *grad_in, lattice_dtype grad_in_dtype,
                                         float *grad_w, float *grad_bias) {
    return resample_backward(coarse, fine, true, grad_out, g_dtype, C_out, w, C_in, dt, in, in_dtype, grad_in,
                             grad_in_dtype, grad_w, grad_bias);
}

// Checks and scratch shared by the Distribute + PointNet forward and backward
// (`out_ok`: the call's own output arguments are valid).
static lattice_status distribute_prepare(lattice *L, const float *pos, const float *feat, int f_d,
                                         const float *params, int n_blocks, const int *widths, const int *groups,
                                         float eps, bool out_ok, const char *what) {
    if (!L) return LATTICE_E_ARG;
    if (!L->splatted) {
        set_err(L, "%s: no lattice yet (call lattice_splat first)", what);
        return LATTICE_E_STATE;
    }
    if (f_d < 0 || L->d + f_d > 16 || (f_d > 0 && L->m > 0 && !feat) || !params || !widths || n_blocks != 3 ||
        widths[0] != 16 || widths[1] != 32 || widths[2] != 64 || (L->m > 0 && !pos) || !out_ok) {
        set_err(L, "%s: bad argument (f_d = %d; the fused PointNet has 3 blocks of widths 16, "
                "32, 64 and d + f_d <= 16)", what, f_d);
        return LATTICE_E_ARG;
    }
    if (groups) {
        const int K[3] = {L->d + f_d, 16, 32};
        for (int l = 0; l < 3; ++l)
            if (groups[l] < 1 || K[l] % groups[l] != 0) {
                set_err(L, "%s: block %d's %d input channels do not split into %d groups", what, l + 1, K[l],
                        groups[l]);
                return LATTICE_E_ARG;
            }
        if (!(eps >= 0.f) || !isfinite(eps)) {
            set_err(L, "%s: eps must be finite and >= 0", what);
            return LATTICE_E_ARG;
        }
    }
    const int64_t E_max = (int64_t)(L->d + 1) * L->max_points;
    if (!L->lvert) {
        bool ok = hipMalloc(&L->lvert, E_max * sizeof(int32_t)) == hipSuccess &&
                  hipMalloc(&L->macc, L->max_vertices * L->d * sizeof(double)) == hipSuccess &&
                  hipMalloc(&L->mu, L->max_vertices * L->d * sizeof(float)) == hipSuccess &&
                  hipMalloc(&L->pn_params, pointnet_padded_count() * sizeof(float)) == hipSuccess &&
                  hipMalloc(&L->pn_keys, (E_max / 64 + 1) * 64 * sizeof(unsigned int)) == hipSuccess;
        if (!ok) {
            (void)hipGetLastError();
            (void)hipFree(L->lvert);
            (void)hipFree(L->macc);
            (void)hipFree(L->mu);
            (void)hipFree(L->pn_params);
            (void)hipFree(L->pn_keys);
            L->lvert = nullptr;
            L->macc = nullptr;
            L->mu = nullptr;
            L->pn_params = nullptr;
            L->pn_keys = nullptr;
            set_err(L, "%s: cannot allocate its scratch", what);
            return LATTICE_E_NOMEM;
        }
    }
    // the normalisation's statistics and affines (1 MiB and 32 KiB)
    if (!L->pn_stats || !L->pn_aff) {
        (void)hipFree(L->pn_stats);
        (void)hipFree(L->pn_aff);
        L->pn_stats = nullptr;
        L->pn_aff = nullptr;
        if (hipMalloc(&L->pn_stats, pointnet_stats_bytes()) != hipSuccess ||
            hipMalloc(&L->pn_aff, pointnet_aff_bytes()) != hipSuccess) {
            (void)hipGetLastError();
            (void)hipFree(L->pn_stats);
            (void)hipFree(L->pn_aff);
            L->pn_stats = nullptr;
            L->pn_aff = nullptr;
            set_err(L, "%s: cannot allocate the normalisation's statistics", what);
            return LATTICE_E_NOMEM;
        }
    }
    return LATTICE_OK;
}

lattice_status lattice_distribute_pointnet(lattice *L, const float *pos, const float *feat, int f_d,
                                           const float *params, int n_blocks, const int *widths, const int *groups,
                                           float eps, void *out, lattice_dtype out_dtype, float *mean) {
    lattice_status s = distribute_prepare(L, pos, feat, f_d, params, n_blocks, widths, groups, eps,
                                          (L && (L->m == 0 || out)) &&
                                              (out_dtype == LATTICE_F32 || out_dtype == LATTICE_BF16),
                                          "distribute_pointnet");
    if (s) return s;
    hipEvent_t t0;
    if ((s = timer_begin(L, LATTICE_STAGE_DISTRIBUTE, &t0))) return s;
    if ((s = check_launch(L, launch_distribute_pointnet(L, pos, feat, f_d, params, groups, eps, out,
                                                        out_dtype == LATTICE_BF16, mean),
                          "distribute_pointnet")))
        return s;
    return timer_end(L, LATTICE_STAGE_DISTRIBUTE, t0);
}

lattice_status lattice_distribute_pointnet_backward(lattice *L, const float *pos, const float *feat, int f_d,
                                                    const float *params, int n_blocks, const int *widths,
                                                    const int *groups, float eps, const float *grad_out,
                                                    float *grad_params) {
    lattice_status s = distribute_prepare(L, pos, feat, f_d, params, n_blocks, widths, groups, eps,
                                          L && grad_params && grad_params != params && (L->m == 0 || grad_out),
                                          "distribute_pointnet_backward");
    if (s) return s;
    if ((s = grow(L, &L->pnb, &L->pnb_bytes, pointnet_backward_scratch_bytes(L), "distribute_pointnet_backward")))
        return s;
    hipEvent_t t0;
    if ((s = timer_begin(L, LATTICE_STAGE_DISTRIBUTE_BACKWARD, &t0))) return s;
    if ((s = check_launch(L, launch_distribute_backward(L, pos, feat, f_d, params, groups, eps, grad_out, grad_params,
                                                        L->pnb),
                          "distribute_pointnet_backward")))
        return s;
    return timer_end(L, LATTICE_STAGE_DISTRIBUTE_BACKWARD, t0);
}

lattice_status lattice_weights_to_bf16(lattice *L, const float *src, int64_t n, uint16_t *dst) {
    if (!L || n < 0 || (n > 0 && (!src || !dst))) return LATTICE_E_ARG;
    return check_launch(L, launch_to_bf16(L, src, n, dst), "to_bf16");
}

static lattice_status read_counters(lattice *L) {
    HIP_TRY(L, hipMemcpyAsync(L->host_counters, L->counters, CNT_WORDS * sizeof(int32_t), hipMemcpyDeviceToHost,
                              L->stream));
    HIP_TRY(L, hipStreamSynchronize(L->stream));
    return LATTICE_OK;
}

static lattice_status device_status(lattice *L) {
    const int st = L->host_counters[CNT_STATUS];
    if (st & ST_CAPACITY) {
        set_err(L, "splat: hash table of %lld slots is full", (long long)L->cap);
        return LATTICE_E_CAPACITY;
    }
    if (st & ST_RANGE) {
        set_err(L, "splat: a key coordinate exceeds +-%d or a batch id is outside [0, 65535]", KEY_MAX);
        return LATTICE_E_RANGE;
    }
    if (st & ST_CLOUDS) {
        set_err(L, "distribute_pointnet: group normalisation keeps per-cloud statistics for batch ids 0..63 only");
        return LATTICE_E_RANGE;
    }
    return LATTICE_OK;
}

lattice_status lattice_num_vertices(lattice *L, int64_t *V) {
    if (!L || !V) return LATTICE_E_ARG;
    *V = 0;
    if (!L->splatted) return LATTICE_E_STATE;
    lattice_status s = read_counters(L);
    if (s) return s;
    *V = L->host_counters[CNT_V];
    return device_status(L);
}

lattice_status lattice_get_status(lattice *L) {
    if (!L) return LATTICE_E_ARG;
    if (!L->splatted) return LATTICE_E_STATE;
    lattice_status s = read_counters(L);
    if (s) return s;
    return device_status(L);
}

lattice_status lattice_get_keys(lattice *L, int32_t *keys, int32_t *batch) {
    if (!L || !keys) return LATTICE_E_ARG;
    if (!L->splatted) return LATTICE_E_STATE;
    return check_launch(L, launch_export_keys(L, keys, batch), "export_keys");
}

lattice_status lattice_get_neighbors(lattice *L, int32_t *nbr) {
    if (!L || !nbr) return LATTICE_E_ARG;
    if (!L->splatted) return LATTICE_E_STATE;
    lattice_status s = ensure_neighbors(L);
    if (s) return s;
    return copy_rows(L, L->nbr, nbr, L->T, -1, L->max_vertices);
}

lattice_status lattice_get_point_simplex(lattice *L, int32_t *idx, float *bary) {
    if (!L) return LATTICE_E_ARG;
    if (!L->splatted) return LATTICE_E_STATE;
    lattice_status s = LATTICE_OK;
    if (idx && L->m > 0) s = copy_rows(L, L->idx, idx, L->d + 1, L->m, L->m);
    if (!s && bary && L->m > 0) s = copy_rows(L, L->bary, bary, L->d + 1, L->m, L->m);
    return s;
}

lattice_status lattice_set_timing(lattice *L, int mode) {
    if (!L || mode < 0 || mode > 2) return LATTICE_E_ARG;
    if (mode == 2) {
        HIP_TRY(L, hipStreamSynchronize(L->stream));
        stage_events *se = events_of(L);
        for (int s = 0; s < LATTICE_NUM_STAGES; ++s) {
            for (auto &pr : se[s].pending) {
                se[s].pool.push_back(pr.first);
                se[s].pool.push_back(pr.second);
            }
            se[s].pending.clear();
            L->timers[s].ms = 0.0;
            L->timers[s].count = 0;
        }
        return LATTICE_OK;
    }
    L->timing = mode;
    return LATTICE_OK;
}

lattice_status lattice_get_timing(lattice *L, double *ms, int64_t *count) {
    if (!L || !ms || !count) return LATTICE_E_ARG;
    HIP_TRY(L, hipStreamSynchronize(L->stream));
    stage_events *se = events_of(L);
    for (int s = 0; s < LATTICE_NUM_STAGES; ++s) {
        for (auto &pr : se[s].pending) {
            float t = 0.f;
            HIP_TRY(L, hipEventElapsedTime(&t, pr.first, pr.second));
            L->timers[s].ms += t;
            L->timers[s].count += 1;
            se[s].pool.push_back(pr.first);
            se[s].pool.push_back(pr.second);
        }
        se[s].pending.clear();
        ms[s] = L->timers[s].ms;
        count[s] = L->timers[s].count;
    }
    return LATTICE_OK;
}

}  // extern "C"
