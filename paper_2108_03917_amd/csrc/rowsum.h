// Column sums of a row-major fp32 matrix of partial results, in a fixed
// order (so that the sums do not depend on scheduling): out[j] = sum over
// r < rows of part[r * n + j].
//
// One level adds each chunk of kRsChunk consecutive rows: a workgroup takes
// 64 columns (one wavefront reads 64 consecutive floats of a row) and splits
// the chunk's rows over its four wavefronts, row r going to wavefront
// r mod 4, each adding its rows in increasing order; the four sums are then
// added in wavefront order.  Chunks are independent workgroups (blockIdx.y),
// and the chunk sums are added by the next level until one row is left.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

// Each source file that includes this gets its own copy of the kernel.
namespace rowsum {
namespace {

constexpr int kRsChunk = 64;
constexpr int kRsBlock = 256;

__global__ __launch_bounds__(kRsBlock) void k_rowsum(const float *__restrict__ part, int64_t rows, int64_t n,
                                                     float *__restrict__ out) {
    __shared__ float red[kRsBlock];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int64_t j = (int64_t)blockIdx.x * 64 + lane;
    const int64_t r0 = (int64_t)blockIdx.y * kRsChunk;
    const int64_t r1 = r0 + kRsChunk < rows ? r0 + kRsChunk : rows;
    float s = 0.f;
    if (j < n)
        for (int64_t r = r0 + w; r < r1; r += 4) s += part[r * n + j];
    red[threadIdx.x] = s;
    __syncthreads();
    if (w == 0 && j < n) out[(int64_t)blockIdx.y * n + j] = ((red[lane] + red[64 + lane]) + red[128 + lane]) + red[192 + lane];
}

// Floats of scratch that sum() needs for `rows` rows of n columns.
inline int64_t scratch_floats(int64_t rows, int64_t n) {
    int64_t total = 0;
    for (int64_t r = rows; r > kRsChunk;) {
        r = (r + kRsChunk - 1) / kRsChunk;
        total += r * n;
    }
    return total;
}

// out[0..n) = column sums of part [rows][n]; `tmp` holds scratch_floats(rows,
// n) floats (the levels' chunk sums).  rows = 0 writes zeros.
inline hipError_t sum(hipStream_t stream, const float *part, int64_t rows, int64_t n, float *tmp, float *out) {
    if (n <= 0) return hipSuccess;
    const unsigned gx = (unsigned)((n + 63) / 64);
    while (rows > kRsChunk) {
        const int64_t chunks = (rows + kRsChunk - 1) / kRsChunk;
        hipLaunchKernelGGL(k_rowsum, dim3(gx, (unsigned)chunks), dim3(kRsBlock), 0, stream, part, rows, n, tmp);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        part = tmp;
        tmp += chunks * n;
        rows = chunks;
    }
    hipLaunchKernelGGL(k_rowsum, dim3(gx, 1), dim3(kRsBlock), 0, stream, part, rows, n, out);
    return hipGetLastError();
}

}  // namespace
}  // namespace rowsum
