// Small data-movement kernels: the x_proj exchange as a sum when all shards share one
// GPU, and the strided row copy the channel splitter (Section IV-B) is built from.
#include "common.h"

namespace ssm {
namespace {

__global__ __launch_bounds__(256) void reduce_add_kernel(float* __restrict__ dst, const float* __restrict__ src,
                                                         int64_t n) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    const int64_t n4 = n / 4;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += stride) {
        float4 a = ((const float4*)dst)[i], b = ((const float4*)src)[i];
        ((float4*)dst)[i] = make_float4(a.x + b.x, a.y + b.y, a.z + b.z, a.w + b.w);
    }
    for (int64_t i = n4 * 4 + (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) dst[i] += src[i];
}

// rows x row_bytes, 16-byte units (all pointers, strides and row_bytes 16-byte aligned)
__global__ __launch_bounds__(256) void copy_rows16_kernel(char* __restrict__ dst, int64_t ld_dst,
                                                          const char* __restrict__ src, int64_t ld_src, int64_t rows,
                                                          int64_t units) {
    const int64_t total = rows * units, stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += stride) {
        const int64_t r = i / units, u = i % units;
        *(uint4*)(dst + r * ld_dst + u * 16) = *(const uint4*)(src + r * ld_src + u * 16);
    }
}

__global__ __launch_bounds__(256) void copy_rows1_kernel(char* __restrict__ dst, int64_t ld_dst,
                                                         const char* __restrict__ src, int64_t ld_src, int64_t rows,
                                                         int64_t row_bytes) {
    const int64_t total = rows * row_bytes, stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += stride) {
        const int64_t r = i / row_bytes, b = i % row_bytes;
        dst[r * ld_dst + b] = src[r * ld_src + b];
    }
}

__global__ __launch_bounds__(256) void fill_zero_kernel(uint32_t* __restrict__ p, int64_t words) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < words; i += stride) p[i] = 0u;
}

unsigned grid_for(int64_t items) { return (unsigned)std::max<int64_t>(1, std::min<int64_t>((items + 255) / 256, 8192)); }

}  // namespace

hipError_t launch_reduce_add(float* dst, const float* src, int64_t n, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    SSM_LAUNCH(reduce_add_kernel, dim3(grid_for((n + 3) / 4)), dim3(256), 0, s, dst, src, n);
    return hipGetLastError();
}

hipError_t launch_fill_zero(void* p, int64_t bytes, hipStream_t s) {
    if (bytes <= 0) return hipSuccess;
    SSM_LAUNCH(fill_zero_kernel, dim3(grid_for(bytes / 4)), dim3(256), 0, s, (uint32_t*)p, bytes / 4);
    return hipGetLastError();
}

hipError_t launch_copy_rows(void* dst, int64_t ld_dst, const void* src, int64_t ld_src, int64_t rows,
                            int64_t row_bytes, hipStream_t s) {
    if (rows <= 0 || row_bytes <= 0) return hipSuccess;
    const bool a16 = ((uintptr_t)dst % 16 == 0) && ((uintptr_t)src % 16 == 0) && ld_dst % 16 == 0 &&
                     ld_src % 16 == 0 && row_bytes % 16 == 0;
    if (a16) {
        SSM_LAUNCH(copy_rows16_kernel, dim3(grid_for(rows * row_bytes / 16)), dim3(256), 0, s, (char*)dst,
                           ld_dst, (const char*)src, ld_src, rows, row_bytes / 16);
    } else {
        SSM_LAUNCH(copy_rows1_kernel, dim3(grid_for(rows * row_bytes)), dim3(256), 0, s, (char*)dst, ld_dst,
                           (const char*)src, ld_src, rows, row_bytes);
    }
    return hipGetLastError();
}

}  // namespace ssm
