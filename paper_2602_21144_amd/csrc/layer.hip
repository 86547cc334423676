// The layer around the mixer shard: the residual stream with its pre-norm (Section II-B:
// the mixer output returns to the residual stream by addition) and Falcon-Mamba's RMS
// norms of the token-dependent fields (Section IV-E: the same selective SSM mixer).
//
// residual_rmsnorm: r = base + (sum of the partial outputs, in order, in fp32); r is
// written to the float32 residual stream and RMSNorm(r) * w to the next mixer's input.
// One workgroup per row; a row of d <= 8192 values stays in registers (8 per thread per
// pass, up to 4 passes), so it is read once and written twice.
//
// bcdt_rms: the reduced x_proj output [delta | B | C] normalised in place, each range by
// its own RMS (no weight). One wave per row.
#include "common.h"

namespace ssm {
namespace {

constexpr int kNormThreads = 256;
constexpr int kNormPasses = 4;   // d <= 8 * 256 * 4

template <typename T> __device__ __forceinline__ void load8(const T* p, float (&v)[8]);
template <> __device__ __forceinline__ void load8<float>(const float* p, float (&v)[8]) {
    const float4 a = *(const float4*)p, b = *(const float4*)(p + 4);
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w; v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}
template <> __device__ __forceinline__ void load8<bf16>(const bf16* p, float (&v)[8]) {
    const bf16x8 a = *(const bf16x8*)p;
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = (float)a[e];
}

template <typename T> __device__ __forceinline__ void store8(T* p, const float (&v)[8]);
template <> __device__ __forceinline__ void store8<float>(float* p, const float (&v)[8]) {
    *(float4*)p = make_float4(v[0], v[1], v[2], v[3]);
    *(float4*)(p + 4) = make_float4(v[4], v[5], v[6], v[7]);
}
template <> __device__ __forceinline__ void store8<bf16>(bf16* p, const float (&v)[8]) {
    bf16x8 a;
#pragma unroll
    for (int e = 0; e < 8; ++e) a[e] = (bf16)v[e];
    *(bf16x8*)p = a;
}

template <typename BT, typename PT, typename OT>
// base may be the residual itself (in place): neither is restrict
__global__ __launch_bounds__(kNormThreads) void residual_rmsnorm_kernel(const BT* base, NormParts parts, float* resid,
                                                                       const float* __restrict__ w, float eps,
                                                                       OT* __restrict__ out, int d) {
    const int64_t row = (int64_t)blockIdx.x * d;
    const int tid = threadIdx.x;
    __shared__ float wsum[kNormThreads / 64];
    float v[kNormPasses][8];
    float ss = 0.0f;
#pragma unroll
    for (int q = 0; q < kNormPasses; ++q) {
        const int c = (q * kNormThreads + tid) * 8;
        if (c < d) {
            load8(base + row + c, v[q]);
            if (parts.n > 0) {
                float s[8];
                load8((const PT*)parts.p[0] + row + c, s);
#pragma unroll
                for (int k = 1; k < kMaxNormParts; ++k) {
                    if (k < parts.n) {
                        float o[8];
                        load8((const PT*)parts.p[k] + row + c, o);
#pragma unroll
                        for (int e = 0; e < 8; ++e) s[e] += o[e];
                    }
                }
#pragma unroll
                for (int e = 0; e < 8; ++e) v[q][e] += s[e];
            }
            store8(resid + row + c, v[q]);
#pragma unroll
            for (int e = 0; e < 8; ++e) ss += v[q][e] * v[q][e];
        }
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) ss += __shfl_xor(ss, off, 64);
    if ((tid & 63) == 0) wsum[tid >> 6] = ss;
    __syncthreads();
    const float tot = (wsum[0] + wsum[1]) + (wsum[2] + wsum[3]);
    const float inv = 1.0f / sqrtf(tot / (float)d + eps);
#pragma unroll
    for (int q = 0; q < kNormPasses; ++q) {
        const int c = (q * kNormThreads + tid) * 8;
        if (c < d) {
            float wv[8], o[8];
            load8(w + c, wv);
#pragma unroll
            for (int e = 0; e < 8; ++e) o[e] = v[q][e] * inv * wv[e];
            store8(out + row + c, o);
        }
    }
}

__global__ __launch_bounds__(256) void bcdt_rms_kernel(float* __restrict__ x, int64_t T, int R, int N, int64_t ld,
                                                       float eps) {
    const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (t >= T) return;   // a whole wave
    const int lane = threadIdx.x & 63, W = R + 2 * N;
    float* row = x + t * ld;
    float s0 = 0.0f, s1 = 0.0f, s2 = 0.0f;
    for (int c = lane; c < W; c += 64) {
        const float v = row[c];
        if (c < R) s0 += v * v;
        else if (c < R + N) s1 += v * v;
        else s2 += v * v;
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        s0 += __shfl_xor(s0, off, 64);
        s1 += __shfl_xor(s1, off, 64);
        s2 += __shfl_xor(s2, off, 64);
    }
    const float i0 = 1.0f / sqrtf(s0 / (float)R + eps), i1 = 1.0f / sqrtf(s1 / (float)N + eps),
                i2 = 1.0f / sqrtf(s2 / (float)N + eps);
    for (int c = lane; c < W; c += 64) row[c] *= (c < R ? i0 : (c < R + N ? i1 : i2));
}

template <typename BT, typename PT, typename OT>
hipError_t norm_launch(const void* base, const NormParts& parts, float* resid, const float* w, float eps, void* out,
                       int64_t T, int d, hipStream_t s) {
    SSM_LAUNCH((residual_rmsnorm_kernel<BT, PT, OT>), dim3((unsigned)T), dim3(kNormThreads), 0, s, (const BT*)base,
               parts, resid, w, eps, (OT*)out, d);
    return hipGetLastError();
}

template <typename BT, typename PT>
hipError_t norm_launch_o(const void* base, const NormParts& parts, float* resid, const float* w, float eps, void* out,
                         bool out_bf16, int64_t T, int d, hipStream_t s) {
    return out_bf16 ? norm_launch<BT, PT, bf16>(base, parts, resid, w, eps, out, T, d, s)
                    : norm_launch<BT, PT, float>(base, parts, resid, w, eps, out, T, d, s);
}

template <typename BT>
hipError_t norm_launch_p(const void* base, const NormParts& parts, bool parts_bf16, float* resid, const float* w,
                         float eps, void* out, bool out_bf16, int64_t T, int d, hipStream_t s) {
    return parts_bf16 ? norm_launch_o<BT, bf16>(base, parts, resid, w, eps, out, out_bf16, T, d, s)
                      : norm_launch_o<BT, float>(base, parts, resid, w, eps, out, out_bf16, T, d, s);
}

}  // namespace

int residual_rmsnorm_max_dim() { return 8 * kNormThreads * kNormPasses; }

hipError_t launch_residual_rmsnorm(const void* base, bool base_bf16, const NormParts& parts, bool parts_bf16,
                                   float* resid, const float* w, float eps, void* out, bool out_bf16, int64_t T, int d,
                                   hipStream_t s) {
    if (T <= 0) return hipSuccess;
    return base_bf16 ? norm_launch_p<bf16>(base, parts, parts_bf16, resid, w, eps, out, out_bf16, T, d, s)
                     : norm_launch_p<float>(base, parts, parts_bf16, resid, w, eps, out, out_bf16, T, d, s);
}

hipError_t launch_bcdt_rms(float* x, int64_t T, int R, int N, int64_t ld, float eps, hipStream_t s) {
    if (T <= 0) return hipSuccess;
    SSM_LAUNCH(bcdt_rms_kernel, dim3((unsigned)((T + 3) / 4)), dim3(256), 0, s, x, T, R, N, ld, eps);
    return hipGetLastError();
}

}  // namespace ssm
