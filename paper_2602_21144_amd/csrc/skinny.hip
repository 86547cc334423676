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

// Epilogue operands of one output element, loaded before the K loop so that their
// latency overlaps the weight stream.
template <int EPI> struct EpiIn {
    __device__ __forceinline__ void load(const SkinnyArgs&, int, int) {}
};

// in_proj: column n < E is channel n of the SSM path (conv window), n >= E the gate.
template <> struct EpiIn<kEpiConv> {
    int slot;
    float w[kMaxConv], hv[kMaxConv - 1], bias;
    __device__ __forceinline__ void load(const SkinnyArgs& p, int m, int n) {
        slot = -1;
        if (n >= p.E) return;
        slot = p.slot[m];
        if (slot < 0 || slot >= p.S) return;
        const int K = p.Kc;
        const bf16* hist = (const bf16*)p.conv_pool + ((int64_t)slot * p.E + n) * (K - 1);
        const bf16* wr = (const bf16*)p.conv_w + (int64_t)n * K;
#pragma unroll
        for (int j = 0; j < kMaxConv; ++j) w[j] = j < K ? (float)wr[j] : 0.0f;
#pragma unroll
        for (int j = 0; j < kMaxConv - 1; ++j) hv[j] = j < K - 1 ? (float)hist[j] : 0.0f;
        bias = (float)((const bf16*)p.conv_b)[n];
    }
    __device__ __forceinline__ void apply(const SkinnyArgs& p, int m, int n, float v) const {
        if (n >= p.E) {
            ((bf16*)p.z)[(int64_t)m * p.ld_z + (n - p.E)] = (bf16)v;
            return;
        }
        if (slot < 0 || slot >= p.S) {
            atomicOr(p.status, SSM_STATUS_BAD_SLOT);
            ((bf16*)p.u)[(int64_t)m * p.E + n] = (bf16)0.0f;
            return;
        }
        const int K = p.Kc;
        const float x = (float)(bf16)v;  // the stored (rounded) projection output enters the window
        float acc = bias;
#pragma unroll
        for (int j = 0; j < kMaxConv - 1; ++j)
            if (j < K - 1) acc += w[j] * hv[j];
        acc += w[K - 1] * x;
        ((bf16*)p.u)[(int64_t)m * p.E + n] = (bf16)silu_f(acc);
        bf16* hist = (bf16*)p.conv_pool + ((int64_t)slot * p.E + n) * (K - 1);
#pragma unroll
        for (int j = 0; j < kMaxConv - 2; ++j)
            if (j < K - 2) hist[j] = (bf16)hv[j + 1];
        if (K > 1) hist[K - 2] = (bf16)x;
    }
};

// dt_proj: one recurrence step of channel n of sequence m on its cached state.
template <> struct EpiIn<kEpiState> {
    int slot;
    float h[kN], a[kN], bc[2 * kN], u, z, bdt, Dn;
    __device__ __forceinline__ void load(const SkinnyArgs& p, int m, int n) {
        slot = p.slot[m];
        if (slot < 0 || slot >= p.S) return;
        const float4* hp = (const float4*)(p.pool + ((int64_t)slot * p.E + n) * kN);
        const float4* al = (const float4*)(p.A_log + (int64_t)n * kN);
        const float4* bt = (const float4*)(p.xdbl + (int64_t)m * p.ld_xdbl + p.R);
#pragma unroll
        for (int q = 0; q < kN / 4; ++q) {
            const float4 hv = hp[q], av = al[q];
            h[4 * q] = hv.x; h[4 * q + 1] = hv.y; h[4 * q + 2] = hv.z; h[4 * q + 3] = hv.w;
            a[4 * q] = av.x; a[4 * q + 1] = av.y; a[4 * q + 2] = av.z; a[4 * q + 3] = av.w;
        }
#pragma unroll
        for (int q = 0; q < 2 * kN / 4; ++q) {
            const float4 bv = bt[q];
            bc[4 * q] = bv.x; bc[4 * q + 1] = bv.y; bc[4 * q + 2] = bv.z; bc[4 * q + 3] = bv.w;
        }
        u = (float)((const bf16*)p.u)[(int64_t)m * p.E + n];
        z = (float)((const bf16*)p.z)[(int64_t)m * p.ld_z + n];
        bdt = p.b_dt[n];
        Dn = p.D[n];
    }
    __device__ __forceinline__ void apply(const SkinnyArgs& p, int m, int n, float v) {
        if (slot < 0 || slot >= p.S) {
            atomicOr(p.status, SSM_STATUS_BAD_SLOT);
            ((bf16*)p.g)[(int64_t)m * p.E + n] = (bf16)0.0f;
            return;
        }
        const float dt = (float)(bf16)v;  // dt is stored in the activation dtype
        const float delta = softplus_f(dt + bdt);
        const float du = delta * u;
        float y = 0.0f;
#pragma unroll
        for (int i = 0; i < kN; ++i) {
            h[i] = fast_exp2(delta * (-__expf(a[i]) * kLog2e)) * h[i] + du * bc[i];
            y += bc[kN + i] * h[i];
        }
        float4* hp = (float4*)(p.pool + ((int64_t)slot * p.E + n) * kN);
#pragma unroll
        for (int q = 0; q < kN / 4; ++q) hp[q] = make_float4(h[4 * q], h[4 * q + 1], h[4 * q + 2], h[4 * q + 3]);
        y += Dn * u;
        ((bf16*)p.g)[(int64_t)m * p.E + n] = (bf16)(y * silu_f(z));
    }
};

// NW waves split K; every thread owns at most one output element of the 16-column tile
// (NW * 64 >= MB * 16), whose epilogue operands it fetches before the K loop. Each wave
// issues the loads of up to KU k-steps (32 each) before its MFMAs.
template <int MB, int NW, int KU, bool A_F32, int EPI>
__global__ __launch_bounds__(NW * 64) void gemm_skinny_kernel(SkinnyArgs p) {
    static_assert(NW * 64 >= MB * 16, "one epilogue element per thread");
    constexpr int MT = MB / 16;
    __shared__ float red[NW][MB * 16];
    const int n0 = blockIdx.x * 16, m0 = blockIdx.y * MB;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;

    const int e = threadIdx.x;
    const int em = m0 + e / 16, en = n0 + (e & 15);
    const bool ework = e < MB * 16 && em < p.M && en < p.N;
    EpiIn<EPI> ein;
    if constexpr (EPI == kEpiConv || EPI == kEpiState) {
        if (ework) ein.load(p, em, en);
    }

    const int ksteps = (p.K + 31) / 32;
    const int per = (ksteps + NW - 1) / NW;
    const int s0 = wave * per, s1 = min(ksteps, s0 + per);
    const int brow = n0 + (lane & 15);
    const int kl = (lane >> 4) * 8;
    const bool bok = brow < p.N;
    f32x4 acc[MT];
#pragma unroll
    for (int i = 0; i < MT; ++i) acc[i] = f32x4{};
    for (int s = s0; s < s1; s += KU) {
        bf16x8 bf[KU], af[KU][MT];
#pragma unroll
        for (int u = 0; u < KU; ++u) {
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
        for (int u = 0; u < KU; ++u)
#pragma unroll
            for (int i = 0; i < MT; ++i) acc[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[u][i], bf[u], acc[i], 0, 0, 0);
    }
    // lane l holds column l % 16 and rows 4 (l / 16) + r of each 16-row tile
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) red[wave][(i * 16 + 4 * (lane >> 4) + r) * 16 + (lane & 15)] = acc[i][r];
    __syncthreads();
    if (!ework) return;
    float v = 0.0f;
#pragma unroll
    for (int w = 0; w < NW; ++w) v += red[w][e];
    if constexpr (EPI == kEpiStoreBf16) ((bf16*)p.C)[(int64_t)em * p.ldc + en] = (bf16)v;
    else if constexpr (EPI == kEpiStoreF32) ((float*)p.C)[(int64_t)em * p.ldc + en] = v;
    else ein.apply(p, em, en, v);
}

template <int MB, int NW, bool AF, int EPI>
void launch_one(const SkinnyArgs& p, dim3 grid, hipStream_t s) {
    // k-steps per wave issued together: bounded by the VGPRs a wave may hold at NW waves
    constexpr int KU = MB <= 16 ? 8 : (MB <= 32 ? 6 : 4);
    SSM_LAUNCH((gemm_skinny_kernel<MB, NW, KU, AF, EPI>), grid, dim3(NW * 64), 0, s, p);
}

template <int MB, bool AF, int EPI>
hipError_t launch_mb(const SkinnyArgs& p, hipStream_t s) {
    const dim3 grid((unsigned)((p.N + 15) / 16), (unsigned)((p.M + MB - 1) / MB));
    // enough waves that each streams at most 8 k-steps, and one thread per output element
    // (the state epilogue keeps a state row per thread: at most 8 waves, 256 VGPRs each)
    const int ksteps = (p.K + 31) / 32;
    constexpr int NWMIN = MB * 16 / 64;
    constexpr int NWMAX = EPI == kEpiState ? 8 : 16;
    const int want = (ksteps + 7) / 8;
    if ((want > 8 || NWMIN > 8) && NWMAX >= 16) launch_one<MB, NWMAX, AF, EPI>(p, grid, s);
    else if (want > 4 || NWMIN > 4) launch_one<MB, (NWMIN > 8 ? NWMAX : 8), AF, EPI>(p, grid, s);
    else launch_one<MB, (NWMIN > 4 ? NWMAX : 4), AF, EPI>(p, grid, s);
    return hipGetLastError();
}

template <bool AF, int EPI>
hipError_t launch_epi(const SkinnyArgs& p, hipStream_t s) {
    if (p.M <= 16) return launch_mb<16, AF, EPI>(p, s);
    // the state epilogue holds a whole state row per thread: at most 32-row tiles (8 waves)
    if (p.M <= 32 || EPI == kEpiState) return launch_mb<32, AF, EPI>(p, s);
    if constexpr (EPI != kEpiState) return launch_mb<64, AF, EPI>(p, s);
    return hipErrorInvalidValue;
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
