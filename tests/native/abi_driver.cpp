// Host-side driver of the C ABI: every entry point of include/lattice.h is
// called on a seeded cloud, in valid and invalid ways, through plain device
// pointers.  Built with AddressSanitizer on the host code only (the device
// code is not instrumented) against a host-instrumented build of the
// library, it checks the library's host code (argument checks, scratch
// growth, caches, timers, destroy) for memory errors.  It checks return
// codes, not numbers: the parity tests do that.  Prints one line per step
// and "abi driver ok" at the end; exits 1 at the first unexpected status.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <random>
#include <vector>

#include "lattice.h"

extern "C" void __lsan_do_leak_check();  // LeakSanitizer's interface (the sanitizer runtime defines it)

namespace {

int failures = 0;

void expect(const char *what, lattice_status got, lattice_status want, const lattice *L = nullptr) {
    std::printf("%-44s %s\n", what, lattice_status_string(got));
    std::fflush(stdout);
    if (got != want) {
        std::printf("  expected %s (%s)\n", lattice_status_string(want), L ? lattice_last_error(L) : "");
        ++failures;
        std::exit(1);
    }
}

template <typename T>
T *dev_alloc(size_t n) {
    T *p = nullptr;
    if (hipMalloc(&p, (n ? n : 1) * sizeof(T)) != hipSuccess) {
        std::printf("hipMalloc failed\n");
        std::exit(1);
    }
    return p;
}

template <typename T>
T *dev_copy(const std::vector<T> &h) {
    T *p = dev_alloc<T>(h.size());
    if (hipMemcpy(p, h.data(), h.size() * sizeof(T), hipMemcpyHostToDevice) != hipSuccess) std::exit(1);
    return p;
}

std::vector<float> normal(size_t n, unsigned seed, float sd = 1.f) {
    std::mt19937 g(seed);
    std::normal_distribution<float> d(0.f, sd);
    std::vector<float> v(n);
    for (auto &x : v) x = d(g);
    return v;
}

}  // namespace

int main() {
    const int d = 3, m = 20000, C = 64, T = LATTICE_TAPS(3);
    std::mt19937 g(7);
    std::uniform_real_distribution<float> u(-1.f, 1.f);
    std::vector<float> hpos((size_t)m * d);
    for (auto &x : hpos) x = u(g);
    float *pos = dev_copy(hpos);
    float *feat = dev_copy(normal((size_t)m * C, 8));
    const float sigma[3] = {0.1f, 0.1f, 0.1f}, sigma2[3] = {0.2f, 0.2f, 0.2f};

    // create: argument errors, then two lattices at 1x and 2x scale
    lattice *L = nullptr, *Lc = nullptr, *bad = nullptr;
    expect("create d = 0", lattice_create(0, sigma, 0.0, m, 0, nullptr, &bad), LATTICE_E_ARG);
    expect("create without out", lattice_create(d, sigma, 0.0, m, 0, nullptr, nullptr), LATTICE_E_ARG);
    expect("create", lattice_create(d, sigma, 0.0, m, 0, nullptr, &L), LATTICE_OK);
    expect("create coarse", lattice_create(d, sigma2, 0.0, m, 0, nullptr, &Lc), LATTICE_OK);
    std::printf("capacity %lld, d %d\n", (long long)lattice_hash_capacity(L), lattice_dim(L));
    const int64_t VM = lattice_max_vertices(L, m);

    expect("conv before splat", lattice_conv(L, feat, LATTICE_F32, C, feat, C, LATTICE_F32, nullptr, feat,
                                             LATTICE_F32), LATTICE_E_STATE, L);
    expect("set_timing 1", lattice_set_timing(L, 1), LATTICE_OK, L);

    // splat, queries
    float *values = dev_alloc<float>((size_t)VM * C);
    uint16_t *values16 = dev_alloc<uint16_t>((size_t)VM * C);
    float *weight = dev_alloc<float>(VM);
    expect("splat bad C", lattice_splat(L, pos, nullptr, m, feat, -1, 0, values, LATTICE_F32, weight), LATTICE_E_ARG, L);
    expect("splat", lattice_splat(L, pos, nullptr, m, feat, C, 0, values, LATTICE_F32, weight), LATTICE_OK, L);
    expect("splat bf16 values", lattice_splat(L, pos, nullptr, m, feat, C, 0, values16, LATTICE_BF16, weight),
           LATTICE_OK, L);
    expect("splat normalised", lattice_splat(L, pos, nullptr, m, feat, C, 1, values, LATTICE_F32, weight),
           LATTICE_OK, L);
    expect("splat coarse (lattice only)", lattice_splat(Lc, pos, nullptr, m, nullptr, 0, 0, nullptr, LATTICE_F32,
                                                        nullptr), LATTICE_OK, Lc);
    int64_t V = 0, Vc = 0;
    expect("num_vertices", lattice_num_vertices(L, &V), LATTICE_OK, L);
    expect("num_vertices coarse", lattice_num_vertices(Lc, &Vc), LATTICE_OK, Lc);
    std::printf("V = %lld, coarse V = %lld\n", (long long)V, (long long)Vc);
    expect("get_status", lattice_get_status(L), LATTICE_OK, L);
    expect("build_neighbors", lattice_build_neighbors(L), LATTICE_OK, L);
    int32_t *keys = dev_alloc<int32_t>((size_t)VM * (d + 1));
    int32_t *nbr = dev_alloc<int32_t>((size_t)VM * T);
    int32_t *sidx = dev_alloc<int32_t>((size_t)m * (d + 1));
    float *sbary = dev_alloc<float>((size_t)m * (d + 1));
    expect("get_keys", lattice_get_keys(L, keys, nullptr), LATTICE_OK, L);
    expect("get_neighbors", lattice_get_neighbors(L, nbr), LATTICE_OK, L);
    expect("get_point_simplex", lattice_get_point_simplex(L, sidx, sbary), LATTICE_OK, L);

    // conv: every path, both compute types, a misaligned output
    float *w32 = dev_copy(normal((size_t)C * T * C, 9, 0.05f));
    uint16_t *w16 = dev_alloc<uint16_t>((size_t)C * T * C);
    float *bias = dev_copy(normal(C, 10));
    float *y = dev_alloc<float>((size_t)VM * C + 4);
    uint16_t *y16 = dev_alloc<uint16_t>((size_t)VM * C);
    expect("weights_to_bf16", lattice_weights_to_bf16(L, w32, (int64_t)C * T * C, w16), LATTICE_OK, L);
    for (int path = 0; path <= 3; ++path) {
        expect("set_conv_path", lattice_set_conv_path(L, path), LATTICE_OK, L);
        expect("conv fp32", lattice_conv(L, values, LATTICE_F32, C, w32, C, LATTICE_F32, bias, y, LATTICE_F32),
               LATTICE_OK, L);
        expect("conv bf16 rows", lattice_conv(L, values16, LATTICE_BF16, C, w16, C, LATTICE_BF16, nullptr, y16,
                                              LATTICE_BF16), LATTICE_OK, L);
    }
    expect("set_conv_path 9", lattice_set_conv_path(L, 9), LATTICE_E_ARG, L);
    expect("conv misaligned out", lattice_conv(L, values, LATTICE_F32, C, w32, C, LATTICE_F32, nullptr, y + 1,
                                               LATTICE_F32), LATTICE_OK, L);
    expect("conv C_in 0", lattice_conv(L, values, LATTICE_F32, 0, w32, C, LATTICE_F32, nullptr, y, LATTICE_F32),
           LATTICE_E_ARG, L);
    expect("conv in == out", lattice_conv(L, values, LATTICE_F32, C, w32, C, LATTICE_F32, nullptr, values,
                                          LATTICE_F32), LATTICE_E_ARG, L);

    // slice, deform slice (with and without the classifier)
    float *sl = dev_alloc<float>((size_t)m * C);
    expect("slice", lattice_slice(L, y, LATTICE_F32, C, sl), LATTICE_OK, L);
    expect("slice bf16", lattice_slice(L, y16, LATTICE_BF16, C, sl), LATTICE_OK, L);
    const int n_cls = 20;
    float *wd = dev_copy(normal(C, 11, 0.1f));
    float *wc = dev_copy(normal((size_t)n_cls * C, 12, 0.1f));
    float *bc = dev_copy(normal(n_cls, 13));
    float *logits = dev_alloc<float>((size_t)m * n_cls);
    float *delta = dev_alloc<float>((size_t)m * (d + 1));
    expect("deform_slice", lattice_deform_slice(L, y, LATTICE_F32, C, wd, 0.1f, nullptr, nullptr, 0, sl, delta),
           LATTICE_OK, L);
    expect("deform_slice + classifier", lattice_deform_slice(L, y, LATTICE_F32, C, wd, 0.1f, wc, bc, n_cls, logits,
                                                             nullptr), LATTICE_OK, L);
    expect("deform_slice n_cls 0", lattice_deform_slice(L, y, LATTICE_F32, C, wd, 0.1f, wc, bc, 0, logits, nullptr),
           LATTICE_E_ARG, L);

    // backward passes
    float *gpoint = dev_copy(normal((size_t)m * C, 14));
    float *glog = dev_copy(normal((size_t)m * n_cls, 15));
    float *gv = dev_alloc<float>((size_t)VM * C);
    float *gx = dev_alloc<float>((size_t)VM * C);
    float *gw = dev_alloc<float>((size_t)C * T * C);
    float *gb = dev_alloc<float>(C);
    float *gfeat = dev_alloc<float>((size_t)m * C);
    float *gwd = dev_alloc<float>(C), *gbd = dev_alloc<float>(1);
    float *gwc = dev_alloc<float>((size_t)n_cls * C), *gbc = dev_alloc<float>(n_cls);
    expect("slice_backward", lattice_slice_backward(L, gpoint, C, gv, LATTICE_F32), LATTICE_OK, L);
    expect("splat_backward", lattice_splat_backward(L, gv, LATTICE_F32, C, 0, nullptr, gfeat), LATTICE_OK, L);
    expect("splat_backward normalised", lattice_splat_backward(L, gv, LATTICE_F32, C, 1, weight, gfeat), LATTICE_OK,
           L);
    expect("conv_backward", lattice_conv_backward(L, gv, LATTICE_F32, C, w32, C, LATTICE_F32, values, LATTICE_F32,
                                                  gx, LATTICE_F32, gw, gb), LATTICE_OK, L);
    expect("conv_backward bf16", lattice_conv_backward(L, gv, LATTICE_F32, C, w16, C, LATTICE_BF16, values,
                                                       LATTICE_F32, gx, LATTICE_F32, gw, gb), LATTICE_OK, L);
    expect("conv_backward_noalloc", lattice_conv_backward_noalloc(L, gv, LATTICE_F32, C, w32, C, LATTICE_F32, values,
                                                                  LATTICE_F32, gx, LATTICE_F32, gw, gb),
           LATTICE_OK, L);
    expect("conv_backward nothing asked", lattice_conv_backward(L, gv, LATTICE_F32, C, w32, C, LATTICE_F32, values,
                                                                LATTICE_F32, nullptr, LATTICE_F32, nullptr, nullptr),
           LATTICE_E_ARG, L);
    expect("deform_slice_backward", lattice_deform_slice_backward(L, y, LATTICE_F32, C, wd, 0.1f, wc, n_cls, glog,
                                                                  gv, LATTICE_F32, gwd, gbd, gwc, gbc), LATTICE_OK, L);
    expect("deform_slice_backward no cls", lattice_deform_slice_backward(L, y, LATTICE_F32, C, wd, 0.1f, nullptr, 0,
                                                                         gpoint, gv, LATTICE_F32, gwd, gbd, nullptr,
                                                                         nullptr), LATTICE_OK, L);

    // down- and upsampling, forward and backward, and the wrong order
    float *yc = dev_alloc<float>((size_t)lattice_max_vertices(Lc, m) * C);
    float *yf = dev_alloc<float>((size_t)VM * C);
    float *gcv = dev_alloc<float>((size_t)lattice_max_vertices(Lc, m) * C);
    expect("downsample", lattice_downsample(L, Lc, values, LATTICE_F32, C, w32, C, LATTICE_F32, bias, yc, LATTICE_F32),
           LATTICE_OK, Lc);
    expect("upsample", lattice_upsample(Lc, L, yc, LATTICE_F32, C, w32, C, LATTICE_F32, nullptr, yf, LATTICE_F32),
           LATTICE_OK, L);
    expect("downsample wrong order", lattice_downsample(Lc, L, yc, LATTICE_F32, C, w32, C, LATTICE_F32, nullptr, yf,
                                                        LATTICE_F32), LATTICE_E_ARG, L);
    expect("downsample_backward", lattice_downsample_backward(L, Lc, yc, LATTICE_F32, C, w32, C, LATTICE_F32, values,
                                                              LATTICE_F32, gx, LATTICE_F32, gw, gb), LATTICE_OK, Lc);
    expect("upsample_backward", lattice_upsample_backward(Lc, L, yf, LATTICE_F32, C, w32, C, LATTICE_F32, yc,
                                                          LATTICE_F32, gcv, LATTICE_F32, gw, gb), LATTICE_OK, L);

    // Distribute + PointNet with group normalisation
    const int f_d = 3, K0 = d + f_d;
    const int widths[3] = {16, 32, 64}, groups[3] = {K0, 16, 32};
    std::vector<float> hp;
    const int K[3] = {K0, 16, 32};
    for (int l = 0; l < 3; ++l) {
        for (int c = 0; c < K[l]; ++c) hp.push_back(1.f);
        for (int c = 0; c < K[l]; ++c) hp.push_back(0.f);
        auto W = normal((size_t)widths[l] * K[l], 20 + l, 0.3f);
        hp.insert(hp.end(), W.begin(), W.end());
        for (int o = 0; o < widths[l]; ++o) hp.push_back(0.01f);
    }
    float *params = dev_copy(hp);
    float *pn = dev_alloc<float>((size_t)VM * 64);
    float *mu = dev_alloc<float>((size_t)VM * d);
    expect("distribute_pointnet", lattice_distribute_pointnet(L, pos, feat, f_d, params, 3, widths, groups, 1e-5f, pn,
                                                              LATTICE_F32, mu), LATTICE_OK, L);
    expect("distribute_pointnet affine", lattice_distribute_pointnet(L, pos, feat, f_d, params, 3, widths, nullptr,
                                                                     0.f, pn, LATTICE_F32, nullptr), LATTICE_OK, L);
    const int bad_widths[3] = {16, 32, 32};
    expect("distribute_pointnet bad widths", lattice_distribute_pointnet(L, pos, feat, f_d, params, 3, bad_widths,
                                                                         groups, 1e-5f, pn, LATTICE_F32, mu),
           LATTICE_E_ARG, L);

    // timers, a re-splat with fewer points, an empty splat
    double ms[LATTICE_NUM_STAGES];
    int64_t cnt[LATTICE_NUM_STAGES];
    expect("get_timing", lattice_get_timing(L, ms, cnt), LATTICE_OK, L);
    for (int s = 0; s < LATTICE_NUM_STAGES; ++s)
        if (cnt[s]) std::printf("  stage %2d: %lld launches, %.3f ms\n", s, (long long)cnt[s], ms[s]);
    expect("set_timing reset", lattice_set_timing(L, 2), LATTICE_OK, L);
    expect("re-splat 1000 points", lattice_splat(L, pos, nullptr, 1000, feat, C, 0, values, LATTICE_F32, weight),
           LATTICE_OK, L);
    expect("conv after re-splat", lattice_conv(L, values, LATTICE_F32, C, w32, C, LATTICE_F32, nullptr, y,
                                               LATTICE_F32), LATTICE_OK, L);
    expect("empty splat", lattice_splat(L, pos, nullptr, 0, nullptr, 0, 0, nullptr, LATTICE_F32, nullptr),
           LATTICE_OK, L);
    expect("num_vertices after empty splat", lattice_num_vertices(L, &V), LATTICE_OK, L);
    expect("hipDeviceSynchronize", hipDeviceSynchronize() == hipSuccess ? LATTICE_OK : LATTICE_E_HIP, LATTICE_OK);

    lattice_destroy(Lc);
    lattice_destroy(L);
    lattice_destroy(nullptr);
    for (void *p : {(void *)pos, (void *)feat, (void *)values, (void *)values16, (void *)weight, (void *)keys,
                    (void *)nbr, (void *)sidx, (void *)sbary, (void *)w32, (void *)w16, (void *)bias, (void *)y,
                    (void *)y16, (void *)sl, (void *)wd, (void *)wc, (void *)bc, (void *)logits, (void *)delta,
                    (void *)gpoint, (void *)glog, (void *)gv, (void *)gx, (void *)gw, (void *)gb, (void *)gfeat,
                    (void *)gwd, (void *)gbd, (void *)gwc, (void *)gbc, (void *)yc, (void *)yf, (void *)gcv,
                    (void *)params, (void *)pn, (void *)mu})
        (void)hipFree(p);
    // The leak check now, then exit without the ROCm runtime's static
    // teardown: under the host sanitizer that teardown trips an allocator
    // check inside the runtime (after every call of this driver has
    // returned), which would hide the driver's own result.
    std::fflush(stdout);
    __lsan_do_leak_check();
    std::printf("abi driver ok\n");
    std::fflush(stdout);
    std::_Exit(failures ? 1 : 0);
}
