// Decode-step projections: C[M][N] = A[M][K] * B[N][K]^T for few rows (one token per
// sequence), where the time is the weight read. Each workgroup owns 16 output columns
// and up to 64 rows; its waves split K, each streaming its share of the 16 weight rows
// with 16-byte loads into v_mfma_f32_16x16x32_bf16, and the partial tiles are summed
// through LDS. Hundreds of workgroups stream disjoint weight rows at once.
//
// Epilogues fuse the per-channel work that follows each projection in a decode step
// (Section IV-A: the cache is read and advanced in place, with no prefix rescan):
//   kEpiConv  (in_proj): SSM-path columns go through the cached conv window + SiLU
//             (window shifted in place), gate-path columns are stored for the gate;
//   kEpiState (dt_proj): Delta = softplus(dt + b_dt), one recurrence step on the cached
//             state in place, D skip and SiLU gate -> g;
//   kEpiStore: plain store (x_proj in fp32, out_proj in bf16).
#include "common.h"

namespace ssm {
namespace {

enum Epi { kEpiStoreBf16 = 0, kEpiStoreF32 = 1, kEpiConv = 2, kEpiState = 3 };

constexpr int kU = 4;  // k-steps (32 each) issued together per wave

template <bool A_F32>
__device__ __forceinline__ bf16x8 load_a(const void* A, int64_t lda, int row, int k) {
    if constexpr (A_F32) {
        const float* p = (const float*)A + (int64_t)row * lda + k;
        const float4 x = *(const float4*)p, y = *(const float4*)(p + 4);
        bf16x8 o;
        o[0] = (bf16)x.x; o[1] = (bf16)x.y; o[2] = (bf16)x.z; o[3] = (bf16)x.w;
        o[4] = (bf16)y.x; o[5] = (bf16)y.y; o[6] = (bf16)y.z; o[7] = (bf16)y.w;
        return o;
    } else {
        return *(const bf16x8*)((const bf16*)A + (int64_t)row * lda + k);
    }
}

// in_proj epilogue: column n < E is channel n of the SSM path, n >= E the gate path.
__device__ __forceinline__ void epi_conv(const SkinnyArgs& p, int m, int n, float v) {
    if (n >= p.E) {
        ((bf16*)p.z)[(int64_t)m * p.ld_z + (n - p.E)] = (bf16)v;
        return;
    }
    const int slot = p.slot[m];
    if (slot < 0 || slot >= p.S) {
        atomicOr(p.status, SSM_STATUS_BAD_SLOT);
        ((bf16*)p.u)[(int64_t)m * p.E + n] = (bf16)0.0f;
        return;
    }
    const int K = p.Kc;
    bf16* hist = (bf16*)p.conv_pool + ((int64_t)slot * p.E + n) * (K - 1);
    const bf16* w = (const bf16*)p.conv_w + (int64_t)n * K;
    const float x = (float)(bf16)v;  // the stored (rounded) projection output enters the window
    float acc = (float)((const bf16*)p.conv_b)[n];
    float hv[kMaxConv];
#pragma unroll
    for (int j = 0; j < kMaxConv - 1; ++j)
        if (j < K - 1) hv[j] = (float)hist[j];
#pragma unroll
    for (int j = 0; j < kMaxConv - 1; ++j)
        if (j < K - 1) acc += (float)w[j] * hv[j];
    acc += (float)w[K - 1] * x;
    ((bf16*)p.u)[(int64_t)m * p.E + n] = (bf16)silu_f(acc);
#pragma unroll
    for (int j = 0; j < kMaxConv - 2; ++j)
        if (j < K - 2) hist[j] = (bf16)hv[j + 1];
    if (K > 1) hist[K - 2] = (bf16)x;
}

// dt_proj epilogue: one recurrence step of channel n of sequence m on its cached state.
__device__ __forceinline__ void epi_state(const SkinnyArgs& p, int m, int n, float v) {
    const int slot = p.slot[m];
    if (slot < 0 || slot >= p.S) {
        atomicOr(p.status, SSM_STATUS_BAD_SLOT);
        ((bf16*)p.g)[(int64_t)m * p.E + n] = (bf16)0.0f;
        return;
    }
    const float dt = (float)(bf16)v;  // dt is stored in the activation dtype
    const float delta = softplus_f(dt + p.b_dt[n]);
    const float u = (float)((const bf16*)p.u)[(int64_t)m * p.E + n];
    const float z = (float)((const bf16*)p.z)[(int64_t)m * p.ld_z + n];
    const float* Bt = p.xdbl + (int64_t)m * p.ld_xdbl + p.R;
    float4* hp = (float4*)(p.pool + ((int64_t)slot * p.E + n) * kN);
    const float4* al = (const float4*)(p.A_log + (int64_t)n * kN);
    const float du = delta * u;
    float y = 0.0f;
#pragma unroll
    for (int q = 0; q < kN / 4; ++q) {
        const float4 h4 = hp[q], a4 = al[q];
        const float4 b4 = *(const float4*)(Bt + 4 * q), c4 = *(const float4*)(Bt + kN + 4 * q);
        float h[4] = {h4.x, h4.y, h4.z, h4.w};
        const float a[4] = {a4.x, a4.y, a4.z, a4.w}, b[4] = {b4.x, b4.y, b4.z, b4.w}, c[4] = {c4.x, c4.y, c4.z, c4.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const float A2 = -__expf(a[i]) * kLog2e;
            h[i] = fast_exp2(delta * A2) * h[i] + du * b[i];
            y += c[i] * h[i];
        }
        hp[q] = make_float4(h[0], h[1], h[2], h[3]);
    }
    y += p.D[n] * u;
    ((bf16*)p.g)[(int64_t)m * p.E + n] = (bf16)(y * silu_f(z));
}

template <int MB, int NW, bool A_F32, int EPI>
__global__ __launch_bounds__(NW * 64) void gemm_skinny_kernel(SkinnyArgs p) {
    constexpr int MT = MB / 16;
    __shared__ float red[NW][MB * 16];
    const int n0 = blockIdx.x * 16, m0 = blockIdx.y * MB;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int ksteps = (p.K + 31) / 32;
    const int per = (ksteps + NW - 1) / NW;
    const int s0 = wave * per, s1 = min(ksteps, s0 + per);
    const int brow = n0 + (lane & 15);
    const int kl = (lane >> 4) * 8;
    const bool bok = brow < p.N;
    f32x4 acc[MT];
#pragma unroll
    for (int i = 0; i < MT; ++i) acc[i] = f32x4{};
    for (int s = s0; s < s1; s += kU) {
        bf16x8 bf[kU], af[kU][MT];
#pragma unroll
        for (int u = 0; u < kU; ++u) {
            const int k = (s + u) * 32 + kl;
            const bool kok = (s + u < s1) && k < p.K;
            bf[u] = (kok && bok) ? *(const bf16x8*)(p.B + (int64_t)brow * p.ldb + k) : bf16x8{};
#pragma unroll
            for (int i = 0; i < MT; ++i) {
                const int arow = m0 + i * 16 + (lane & 15);
                af[u][i] = (kok && arow < p.M) ? load_a<A_F32>(p.A, p.lda, arow, k) : bf16x8{};
            }
        }
#pragma unroll
        for (int u = 0; u < kU; ++u)
#pragma unroll
            for (int i = 0; i < MT; ++i) acc[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[u][i], bf[u], acc[i], 0, 0, 0);
    }
    // lane l holds column l % 16 and rows 4 (l / 16) + r of each 16-row tile
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) red[wave][(i * 16 + 4 * (lane >> 4) + r) * 16 + (lane & 15)] = acc[i][r];
    __syncthreads();
    for (int e = threadIdx.x; e < MB * 16; e += NW * 64) {
        const int m = m0 + e / 16, n = n0 + (e & 15);
        if (m >= p.M || n >= p.N) continue;
        float v = 0.0f;
#pragma unroll
        for (int w = 0; w < NW; ++w) v += red[w][e];
        if constexpr (EPI == kEpiStoreBf16) ((bf16*)p.C)[(int64_t)m * p.ldc + n] = (bf16)v;
        else if constexpr (EPI == kEpiStoreF32) ((float*)p.C)[(int64_t)m * p.ldc + n] = v;
        else if constexpr (EPI == kEpiConv) epi_conv(p, m, n, v);
        else epi_state(p, m, n, v);
    }
}

template <int MB, bool AF, int EPI>
hipError_t launch_mb(const SkinnyArgs& p, hipStream_t s) {
    const dim3 grid((unsigned)((p.N + 15) / 16), (unsigned)((p.M + MB - 1) / MB));
    // waves per workgroup: enough that each streams about 8 k-steps of 32
    const int ksteps = (p.K + 31) / 32;
    if (ksteps >= 96) hipLaunchKernelGGL((gemm_skinny_kernel<MB, 16, AF, EPI>), grid, dim3(1024), 0, s, p);
    else if (ksteps >= 48) hipLaunchKernelGGL((gemm_skinny_kernel<MB, 8, AF, EPI>), grid, dim3(512), 0, s, p);
    else if (ksteps >= 16) hipLaunchKernelGGL((gemm_skinny_kernel<MB, 4, AF, EPI>), grid, dim3(256), 0, s, p);
    else hipLaunchKernelGGL((gemm_skinny_kernel<MB, 2, AF, EPI>), grid, dim3(128), 0, s, p);
    return hipGetLastError();
}

template <bool AF, int EPI>
hipError_t launch_epi(const SkinnyArgs& p, hipStream_t s) {
    if (p.M <= 16) return launch_mb<16, AF, EPI>(p, s);
    if (p.M <= 32) return launch_mb<32, AF, EPI>(p, s);
    return launch_mb<64, AF, EPI>(p, s);
}

}  // namespace

hipError_t launch_gemm_skinny(const SkinnyArgs& p, SkinnyEpi epi, hipStream_t s) {
    if (p.M <= 0 || p.N <= 0) return hipSuccess;
    switch (epi) {
        case kSkinnyStoreBf16: return p.a_f32 ? launch_epi<true, kEpiStoreBf16>(p, s) : launch_epi<false, kEpiStoreBf16>(p, s);
        case kSkinnyStoreF32: return p.a_f32 ? launch_epi<true, kEpiStoreF32>(p, s) : launch_epi<false, kEpiStoreF32>(p, s);
        case kSkinnyConv: return launch_epi<false, kEpiConv>(p, s);
        case kSkinnyState: return launch_epi<true, kEpiState>(p, s);
    }
    return hipErrorInvalidValue;
}

}  // namespace ssm
