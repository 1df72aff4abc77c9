// Row l2 normalisation and its backward (gfx950).
//
// Sec. 3.1 ("Normalizing Attention", eq. normalized-yoso): N-YOSO returns the
// attention output with every row scaled to unit length, l2(B V).  Sec. 4 (the
// opening of the experiments): queries and keys are l2-normalised before they are
// hashed.  Both are the same row operation
//   y = x / ||x||                       (y = 0 for a zero row)
// with the Jacobian-vector product
//   dx = (dy - y (y . dy)) / ||x||      (dx = 0 for a zero row).
// The backward recomputes ||x|| and y from x instead of reading a stored y, so it
// needs no extra buffer and is exact for bf16 inputs too.
//
// Both kernels are HBM-bound streams: 16 lanes per 64-value row (16 bytes of fp32
// or 8 bytes of bf16 each), the row sums by a 16-lane butterfly, every row read
// and written once.  Arithmetic is fp32; the norm is sqrt of the fp32 sum of
// squares (correctly rounded square root and division).
#include "common.h"
#include "launch.h"
#include "timing.h"

namespace yoso {

namespace {

constexpr int kNormThreads = 256;

template <bool BF16>
__device__ __forceinline__ void load4(const void *base, int64_t off, float v[4]) {
    if constexpr (BF16) {
        const uint2 w = *reinterpret_cast<const uint2 *>(static_cast<const uint16_t *>(base) + off);
        v[0] = __uint_as_float(w.x << 16);
        v[1] = __uint_as_float(w.x & 0xFFFF0000u);
        v[2] = __uint_as_float(w.y << 16);
        v[3] = __uint_as_float(w.y & 0xFFFF0000u);
    } else {
        const float4 w = *reinterpret_cast<const float4 *>(static_cast<const float *>(base) + off);
        v[0] = w.x; v[1] = w.y; v[2] = w.z; v[3] = w.w;
    }
}

template <bool BF16>
__device__ __forceinline__ void store4(void *base, int64_t off, const float v[4]) {
    if constexpr (BF16) {
        uint2 w;
        w.x = static_cast<uint32_t>(f32_to_bf16(v[0])) | (static_cast<uint32_t>(f32_to_bf16(v[1])) << 16);
        w.y = static_cast<uint32_t>(f32_to_bf16(v[2])) | (static_cast<uint32_t>(f32_to_bf16(v[3])) << 16);
        *reinterpret_cast<uint2 *>(static_cast<uint16_t *>(base) + off) = w;
    } else {
        *reinterpret_cast<float4 *>(static_cast<float *>(base) + off) = make_float4(v[0], v[1], v[2], v[3]);
    }
}

// One row per 16 lanes, grid-stride.  Every lane of a row group runs the same
// number of iterations (the row index is uniform across the group), so the
// butterfly always runs with the whole group active.
template <bool BF16>
__global__ __launch_bounds__(kNormThreads) void l2norm_kernel(const void *__restrict__ x, void *__restrict__ y,
                                                              int64_t rows) {
    const int q = threadIdx.x & 15;
    const int64_t stride = static_cast<int64_t>(gridDim.x) * (kNormThreads / 16);
    for (int64_t r = (static_cast<int64_t>(blockIdx.x) * kNormThreads + threadIdx.x) >> 4; r < rows; r += stride) {
        float v[4];
        load4<BF16>(x, r * D + 4 * q, v);
        const float ss = group_sum(v[0] * v[0] + v[1] * v[1] + v[2] * v[2] + v[3] * v[3], 16);
        const float nrm = sqrtf(ss);
#pragma unroll
        for (int i = 0; i < 4; i++) v[i] = nrm > 0.f ? v[i] / nrm : 0.f;
        store4<BF16>(y, r * D + 4 * q, v);
    }
}

template <bool BF16>
__global__ __launch_bounds__(kNormThreads) void l2norm_bwd_kernel(const void *__restrict__ x,
                                                                  const void *__restrict__ dy,
                                                                  void *__restrict__ dx, int64_t rows) {
    const int q = threadIdx.x & 15;
    const int64_t stride = static_cast<int64_t>(gridDim.x) * (kNormThreads / 16);
    for (int64_t r = (static_cast<int64_t>(blockIdx.x) * kNormThreads + threadIdx.x) >> 4; r < rows; r += stride) {
        float v[4], g[4];
        load4<BF16>(x, r * D + 4 * q, v);
        load4<BF16>(dy, r * D + 4 * q, g);
        const float ss = group_sum(v[0] * v[0] + v[1] * v[1] + v[2] * v[2] + v[3] * v[3], 16);
        const float nrm = sqrtf(ss);
        float u[4];
#pragma unroll
        for (int i = 0; i < 4; i++) u[i] = nrm > 0.f ? v[i] / nrm : 0.f;
        const float t = group_sum(u[0] * g[0] + u[1] * g[1] + u[2] * g[2] + u[3] * g[3], 16);
        float o[4];
#pragma unroll
        for (int i = 0; i < 4; i++) o[i] = nrm > 0.f ? (g[i] - u[i] * t) / nrm : 0.f;
        store4<BF16>(dx, r * D + 4 * q, o);
    }
}

unsigned norm_grid(int64_t rows) {
    const int64_t blocks = (rows * 16 + kNormThreads - 1) / kNormThreads;
    return static_cast<unsigned>(blocks < 8192 ? (blocks > 0 ? blocks : 1) : 8192);
}

}  // namespace

hipError_t launch_l2norm(const void *x, void *y, bool bf16, int64_t rows, hipStream_t stream) {
    if (rows == 0) return hipSuccess;
    KernelTimer timer("l2norm_kernel", stream);
    if (bf16)
        hipLaunchKernelGGL(l2norm_kernel<true>, dim3(norm_grid(rows)), dim3(kNormThreads), 0, stream, x, y, rows);
    else
        hipLaunchKernelGGL(l2norm_kernel<false>, dim3(norm_grid(rows)), dim3(kNormThreads), 0, stream, x, y, rows);
    return hipGetLastError();
}

hipError_t launch_l2norm_backward(const void *x, const void *dy, void *dx, bool bf16, int64_t rows,
                                  hipStream_t stream) {
    if (rows == 0) return hipSuccess;
    KernelTimer timer("l2norm_bwd_kernel", stream);
    if (bf16)
        hipLaunchKernelGGL(l2norm_bwd_kernel<true>, dim3(norm_grid(rows)), dim3(kNormThreads), 0, stream, x, dy,
                           dx, rows);
    else
        hipLaunchKernelGGL(l2norm_bwd_kernel<false>, dim3(norm_grid(rows)), dim3(kNormThreads), 0, stream, x, dy,
                           dx, rows);
    return hipGetLastError();
}

}  // namespace yoso
