// Measurement aid, built as its own executable (not part of liblattice):
// the sustained rates of the chip that the kernels' roofline fractions are
// read against.
//
//   mfma_f32   v_mfma_f32_32x32x2f32 in a loop, NACC independent accumulators
//              per wavefront, no memory traffic inside the loop
//   mfma_bf16  v_mfma_f32_32x32x16_bf16, the same way
//   copy       a float4 grid-stride copy of `bytes` bytes (read + write)
//   read       a float4 grid-stride sum of `bytes` bytes (read only)
//
// Each case is launched once untimed, then timed with HIP events over REPS
// launches; one JSON line per case on stdout.  The copy is also the kernel
// whose FETCH_SIZE and WRITE_SIZE counters calibrate the traffic figures.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdio>
#include <cstdlib>

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

#define CHECK(x)                                                                          \
    do {                                                                                  \
        hipError_t e_ = (x);                                                              \
        if (e_ != hipSuccess) {                                                           \
            fprintf(stderr, "%s:%d %s: %s\n", __FILE__, __LINE__, #x, hipGetErrorString(e_)); \
            exit(1);                                                                      \
        }                                                                                 \
    } while (0)

constexpr int kBlock = 256;

template <int NACC>
__global__ __launch_bounds__(kBlock) void k_mfma_f32(float *out, int iters) {
    f32x16_t acc[NACC];
#pragma unroll
    for (int j = 0; j < NACC; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[j][r] = 0.f;
    const float a = threadIdx.x * 1e-3f, b = 1.0f;
    for (int i = 0; i < iters; ++i)
#pragma unroll
        for (int j = 0; j < NACC; ++j) acc[j] = __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, acc[j], 0, 0, 0);
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < NACC; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) s += acc[j][r];
    out[(int64_t)blockIdx.x * kBlock + threadIdx.x] = s;
}

template <int NACC>
__global__ __launch_bounds__(kBlock) void k_mfma_bf16(float *out, int iters) {
    f32x16_t acc[NACC];
#pragma unroll
    for (int j = 0; j < NACC; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[j][r] = 0.f;
    bf16x8_t a, b;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        a[i] = (__bf16)(threadIdx.x * 1e-3f);
        b[i] = (__bf16)1.0f;
    }
    for (int i = 0; i < iters; ++i)
#pragma unroll
        for (int j = 0; j < NACC; ++j) acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[j], 0, 0, 0);
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < NACC; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) s += acc[j][r];
    out[(int64_t)blockIdx.x * kBlock + threadIdx.x] = s;
}

__global__ __launch_bounds__(kBlock) void k_copy(const float4 *__restrict__ src, float4 *__restrict__ dst, int64_t n) {
    const int64_t stride = (int64_t)gridDim.x * kBlock;
    for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < n; i += stride) dst[i] = src[i];
}

__global__ __launch_bounds__(kBlock) void k_read(const float4 *__restrict__ src, int64_t n, float *out) {
    const int64_t stride = (int64_t)gridDim.x * kBlock;
    float s = 0.f;
    for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < n; i += stride) {
        const float4 v = src[i];
        s += (v.x + v.y) + (v.z + v.w);
    }
    // a sum that is never zero for these inputs keeps the loads alive; one
    // store per thread
    out[(int64_t)blockIdx.x * kBlock + threadIdx.x] = s;
}

// Milliseconds per launch of f over reps launches (one untimed launch first).
template <typename F>
static float time_ms(F f, int reps) {
    f();
    CHECK(hipDeviceSynchronize());
    hipEvent_t e0, e1;
    CHECK(hipEventCreate(&e0));
    CHECK(hipEventCreate(&e1));
    CHECK(hipEventRecord(e0, 0));
    for (int i = 0; i < reps; ++i) f();
    CHECK(hipEventRecord(e1, 0));
    CHECK(hipEventSynchronize(e1));
    CHECK(hipGetLastError());
    float ms = 0.f;
    CHECK(hipEventElapsedTime(&ms, e0, e1));
    CHECK(hipEventDestroy(e0));
    CHECK(hipEventDestroy(e1));
    return ms / reps;
}

int main(int argc, char **argv) {
    const int64_t mib = argc > 1 ? atoll(argv[1]) : 1024;  // bytes copied / read per launch, MiB
    const int iters = 20000;
    const int reps = 5;
    hipDeviceProp_t prop;
    CHECK(hipGetDeviceProperties(&prop, 0));
    const int cus = prop.multiProcessorCount;

    const int max_blocks = 32 * cus;
    float *out;
    CHECK(hipMalloc(&out, (size_t)max_blocks * kBlock * sizeof(float)));
    for (int per_cu : {1, 2, 4}) {
        const int blocks = per_cu * cus;
        const double waves = (double)blocks * (kBlock / 64);
        {
            const float ms = time_ms([&] { hipLaunchKernelGGL(k_mfma_f32<4>, dim3(blocks), dim3(kBlock), 0, 0, out, iters); }, reps);
            const double flops = waves * iters * 4 * (32.0 * 32 * 2 * 2);
            printf("{\"case\": \"mfma_f32_32x32x2\", \"workgroups_per_cu\": %d, \"acc_per_wave\": 4, \"us\": %.1f, \"tflops\": %.1f}\n",
                   per_cu, ms * 1e3, flops / (ms * 1e-3) / 1e12);
        }
        {
            const float ms = time_ms([&] { hipLaunchKernelGGL(k_mfma_bf16<4>, dim3(blocks), dim3(kBlock), 0, 0, out, iters); }, reps);
            const double flops = waves * iters * 4 * (32.0 * 32 * 16 * 2);
            printf("{\"case\": \"mfma_bf16_32x32x16\", \"workgroups_per_cu\": %d, \"acc_per_wave\": 4, \"us\": %.1f, \"tflops\": %.1f}\n",
                   per_cu, ms * 1e3, flops / (ms * 1e-3) / 1e12);
        }
    }
    fflush(stdout);

    const int64_t bytes = mib << 20;
    const int64_t n4 = bytes / 16;
    float4 *src, *dst;
    CHECK(hipMalloc(&src, (size_t)bytes));
    CHECK(hipMalloc(&dst, (size_t)bytes));
    CHECK(hipMemset(src, 0x3c, (size_t)bytes));  // 0x3c3c3c3c: about 0.0115 as fp32
    for (int per_cu : {1, 2, 4, 8, 16, 32}) {
        const int blocks = per_cu * cus;
        const float ms = time_ms([&] { hipLaunchKernelGGL(k_copy, dim3(blocks), dim3(kBlock), 0, 0, src, dst, n4); }, reps);
        printf("{\"case\": \"copy\", \"mib\": %lld, \"workgroups_per_cu\": %d, \"us\": %.1f, \"gbs_read_plus_write\": %.1f}\n",
               (long long)mib, per_cu, ms * 1e3, 2.0 * bytes / (ms * 1e-3) / 1e9);
    }
    for (int per_cu : {1, 2, 4, 8, 16, 32}) {
        const int blocks = per_cu * cus;
        const float ms = time_ms([&] { hipLaunchKernelGGL(k_read, dim3(blocks), dim3(kBlock), 0, 0, src, n4, out); }, reps);
        printf("{\"case\": \"read\", \"mib\": %lld, \"workgroups_per_cu\": %d, \"us\": %.1f, \"gbs\": %.1f}\n",
               (long long)mib, per_cu, ms * 1e3, 1.0 * bytes / (ms * 1e-3) / 1e9);
    }
    CHECK(hipFree(src));
    CHECK(hipFree(dst));
    CHECK(hipFree(out));
    return 0;
}
