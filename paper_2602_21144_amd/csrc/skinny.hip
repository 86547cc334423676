// Decode-step projections: C[M][N] = A[M][K] * B[N][K]^T for few rows (one token per
// sequence), where the time is the weight read. Each workgroup owns 16 output columns;
// its waves split K and the partial tiles are summed through LDS. Hundreds of workgroups
// stream disjoint weight rows at once. Two ways of moving the operands:
//   - streamed (up to 16 rows, bf16, K a multiple of 64: in_proj, x_proj, out_proj of a
//     decode step): whole-line loads into registers, re-laid out through LDS as MFMA
//     fragments (gemm_gemv_kernel);
//   - direct (up to 64 rows, any K, fp32 activations): 16-byte fragment loads straight
//     into v_mfma_f32_16x16x32_bf16 (gemm_skinny_kernel); for 17..64 bf16 rows over wide
//     outputs, 32 columns per workgroup (gemm_skinny32_kernel), which halves the
//     activation re-reads.
// The streamed kernel can also apply Mamba-2's gated RMSNorm to its activations as they
// are loaded (out_proj of a Mamba-2 decode step).
//
// Epilogues fuse the per-channel work that follows each projection in a decode step
// (Section IV-A: the cache is read and advanced in place, with no prefix rescan):
//   kEpiConv  (in_proj): conv-path columns go through the cached conv window + SiLU
//             (window shifted in place), the other columns (gate, Mamba-2's dt) are stored;
//   kEpiState (dt_proj): Delta = softplus(dt + b_dt), one recurrence step on the cached
//             state in place, D skip and SiLU gate -> g;
//   kEpiStore: plain store (x_proj in fp32, out_proj in bf16).
#include "common.h"

namespace ssm {
namespace {

enum Epi { kEpiStoreBf16 = 0, kEpiStoreF32 = 1, kEpiConv = 2, kEpiState = 3 };

// An A fragment as loaded: 8 bf16, or 8 fp32 rounded to bf16 when it enters the MFMA.
template <bool A_F32> struct ARaw {
    u32x4 v;
    __device__ __forceinline__ void load(__amdgpu_buffer_rsrc_t r, uint32_t off) { v = buffer_load16(r, off); }
    __device__ __forceinline__ bf16x8 get() const { return __builtin_bit_cast(bf16x8, v); }
};
template <> struct ARaw<true> {
    u32x4 v0, v1;
    __device__ __forceinline__ void load(__amdgpu_buffer_rsrc_t r, uint32_t off) {
        v0 = buffer_load16(r, off);
        v1 = buffer_load16(r, off == kOffOutOfRange ? off : off + 16);
    }
    __device__ __forceinline__ bf16x8 get() const {
        const f32x4 x = __builtin_bit_cast(f32x4, v0), y = __builtin_bit_cast(f32x4, v1);
        bf16x8 o;
        o[0] = (bf16)x[0]; o[1] = (bf16)x[1]; o[2] = (bf16)x[2]; o[3] = (bf16)x[3];
        o[4] = (bf16)y[0]; o[5] = (bf16)y[1]; o[6] = (bf16)y[2]; o[7] = (bf16)y[3];
        return o;
    }
};

// Epilogue operands of one output element. load_slot() issues the cache-slot index
// before the weight loads; load() issues the operands (some addressed by that slot)
// right after them, so that the slot's latency, the weight stream and the operand
// fetch overlap. Both are branch-free: every thread loads from in-range (clamped)
// rows, slots and taps, and apply() decides what the values mean, so the compiler
// keeps all of these loads in flight together.
template <int EPI> struct EpiIn {
    __device__ __forceinline__ void load_slot(const SkinnyArgs&, int) {}
    __device__ __forceinline__ void load(const SkinnyArgs&, int, int) {}
};

__device__ __forceinline__ bool slot_ok(int slot, int S) { return slot >= 0 && slot < S; }

// in_proj: column n in [conv_lo, conv_lo + conv_n) is channel n - conv_lo of the conv path
// (Mamba: the SSM half; Mamba-2: x, B and C), every other column is stored as it is.
// Needs 2 <= d_conv <= 4 (at least one cached tap).
template <> struct EpiIn<kEpiConv> {
    int slot;
    float w[kMaxConv], hv[kMaxConv - 1], bias, wlast;  // wlast = w[K - 1], the current token's tap
    __device__ __forceinline__ void load_slot(const SkinnyArgs& p, int m) { slot = p.slot[m]; }
    __device__ __forceinline__ void load(const SkinnyArgs& p, int, int n) {
        const int K = p.Kc;
        const int c = n - p.conv_lo;
        const int cc = c >= 0 && c < p.conv_n ? c : 0;  // stored columns read channel 0 and ignore it
        const int sc = slot_ok(slot, p.S) ? slot : 0;
        const bf16* hist = (const bf16*)p.conv_pool + ((int64_t)sc * p.conv_n + cc) * (K - 1);
        const bf16* wr = (const bf16*)p.conv_w + (int64_t)cc * K;
#pragma unroll
        for (int j = 0; j < kMaxConv; ++j) w[j] = (float)wr[j < K ? j : K - 1];
#pragma unroll
        for (int j = 0; j < kMaxConv - 1; ++j) hv[j] = (float)hist[j < K - 1 ? j : K - 2];
        bias = (float)((const bf16*)p.conv_b)[cc];
        wlast = 0.0f;
#pragma unroll
        for (int j = 0; j < kMaxConv; ++j) {
            if (j == K - 1) wlast = w[j];  // static indices only: the arrays stay in registers
            w[j] = j < K ? w[j] : 0.0f;
        }
#pragma unroll
        for (int j = 0; j < kMaxConv - 1; ++j) hv[j] = j < K - 1 ? hv[j] : 0.0f;
    }
    __device__ __forceinline__ void apply(const SkinnyArgs& p, int m, int n, float v) const {
        const int c = n - p.conv_lo;
        if (c < 0 || c >= p.conv_n) {
            ((bf16*)p.C)[(int64_t)m * p.ldc + n] = (bf16)v;
            return;
        }
        bf16* u = (bf16*)p.u + (int64_t)m * p.conv_n + c;
        if (!slot_ok(slot, p.S)) {
            atomicOr(p.status, SSM_STATUS_BAD_SLOT);
            *u = (bf16)0.0f;
            return;
        }
        const int K = p.Kc;
        const float x = (float)(bf16)v;  // the stored (rounded) projection output enters the window
        float acc = bias;
#pragma unroll
        for (int j = 0; j < kMaxConv - 1; ++j)
            if (j < K - 1) acc += w[j] * hv[j];
        acc += wlast * x;
        *u = (bf16)silu_f(acc);
        bf16* hist = (bf16*)p.conv_pool + ((int64_t)slot * p.conv_n + c) * (K - 1);
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
    __device__ __forceinline__ void load_slot(const SkinnyArgs& p, int m) { slot = p.slot[m]; }
    __device__ __forceinline__ void load(const SkinnyArgs& p, int m, int n) {
        const int sc = slot_ok(slot, p.S) ? slot : 0;
        const float4* hp = (const float4*)(p.pool + ((int64_t)sc * p.E + n) * kN);
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
        if (!slot_ok(slot, p.S)) {
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
// (NW * 64 >= MB * 16). Each wave issues the loads of up to KU k-steps (32 each) before
// its MFMAs; the first batch goes out right after the epilogue's slot index and before
// the epilogue operands.
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
    const int emc = em < p.M ? em : p.M - 1, enc = en < p.N ? en : p.N - 1;  // in-range for the fetch
    EpiIn<EPI> ein;
    ein.load_slot(p, emc);

    const int ksteps = (p.K + 31) / 32;
    const int per = (ksteps + NW - 1) / NW;
    const int s0 = wave * per, s1 = min(ksteps, s0 + per);
    const int kl = (lane >> 4) * 8;
    // the tile's weight rows and activation rows as buffer resources: rows past N or M
    // lie outside them and read as zero, as do k-steps outside this wave's share
    constexpr int asz = A_F32 ? 4 : 2;
    const __amdgpu_buffer_rsrc_t rb =
        buffer_rsrc(p.B + (int64_t)n0 * p.ldb, (uint32_t)(min(16, p.N - n0) * p.ldb * 2));
    const __amdgpu_buffer_rsrc_t ra = buffer_rsrc((const char*)p.A + (int64_t)m0 * p.lda * asz,
                                                  (uint32_t)(min(MB, p.M - m0) * p.lda * asz));
    f32x4 acc[MT];
#pragma unroll
    for (int i = 0; i < MT; ++i) acc[i] = f32x4{};
    u32x4 bf[KU];
    ARaw<A_F32> af[KU][MT];
    auto load_batch = [&](int s) {
#pragma unroll
        for (int u = 0; u < KU; ++u) {
            const int k = (s + u) * 32 + kl;
            const bool kok = (s + u < s1) && k < p.K;
            bf[u] = buffer_load16(rb, kok ? (uint32_t)(((lane & 15) * p.ldb + k) * 2) : kOffOutOfRange);
#pragma unroll
            for (int i = 0; i < MT; ++i)
                af[u][i].load(ra, kok ? (uint32_t)(((i * 16 + (lane & 15)) * p.lda + k) * asz) : kOffOutOfRange);
        }
    };
    auto mma_batch = [&]() {
#pragma unroll
        for (int u = 0; u < KU; ++u)
#pragma unroll
            for (int i = 0; i < MT; ++i)
                acc[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[u][i].get(), __builtin_bit_cast(bf16x8, bf[u]),
                                                                 acc[i], 0, 0, 0);
    };
    load_batch(s0);
    // keep the order: weights in flight, then the slot-addressed epilogue fetch (which waits
    // only for the slot index), then the MFMAs (which wait for the weights)
    __builtin_amdgcn_sched_barrier(0);
    ein.load(p, emc, enc);
    __builtin_amdgcn_sched_barrier(0);
    mma_batch();
    for (int s = s0 + KU; s < s1; s += KU) {
        load_batch(s);
        mma_batch();
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

// 17 to 64 rows: the fragment kernel with 32 output columns per workgroup. Every
// workgroup reads all MB activation rows, so halving the number of column tiles halves
// those re-reads (the 3584-wide in_proj of 64 sequences read ~205 MB of activations from
// L2 on 16-column tiles). NW waves split K; each k-step loads two weight fragments (rows
// n0 + 16 j) and the MT activation fragments and issues 2 MT MFMAs. The waves' partial
// tiles meet in LDS; each thread then finishes EPT output elements. Plain stores and the
// conv epilogue only (the state epilogue holds a whole state row per element).
template <int MB, int NW, int KU, int EPI>
__global__ __launch_bounds__(NW * 64) void gemm_skinny32_kernel(SkinnyArgs p) {
    constexpr int MT = MB / 16, NB = 32;
    constexpr int EPT = MB * NB / (NW * 64);
    static_assert(EPT * NW * 64 == MB * NB, "whole elements per thread");
    __shared__ float red[NW][MB * NB];
    const int n0 = blockIdx.x * NB, m0 = blockIdx.y * MB;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;

    // epilogue elements of this thread: e = tid + t NW 64, row e / 32, column e % 32
    EpiIn<EPI> ein[EPT];
    int em[EPT], en[EPT];
#pragma unroll
    for (int t = 0; t < EPT; ++t) {
        const int e = threadIdx.x + t * NW * 64;
        em[t] = m0 + e / NB;
        en[t] = n0 + e % NB;
        ein[t].load_slot(p, em[t] < p.M ? em[t] : p.M - 1);
    }

    const int ksteps = (p.K + 31) / 32;
    const int per = (ksteps + NW - 1) / NW;
    const int s0 = wave * per, s1 = min(ksteps, s0 + per);
    const int kl = (lane >> 4) * 8;
    // weight rows past N and activation rows past M lie outside the resources: zeros
    const __amdgpu_buffer_rsrc_t rb = buffer_rsrc(p.B + (int64_t)n0 * p.ldb, (uint32_t)(min(NB, p.N - n0) * p.ldb * 2));
    const __amdgpu_buffer_rsrc_t ra = buffer_rsrc((const bf16*)p.A + (int64_t)m0 * p.lda,
                                                  (uint32_t)(min(MB, p.M - m0) * p.lda * 2));
    f32x4 acc[2][MT];
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int i = 0; i < MT; ++i) acc[j][i] = f32x4{};
    u32x4 bf[KU][2], af[KU][MT];
    auto load_batch = [&](int s) {
#pragma unroll
        for (int u = 0; u < KU; ++u) {
            const int k = (s + u) * 32 + kl;
            const bool kok = (s + u < s1) && k < p.K;
#pragma unroll
            for (int j = 0; j < 2; ++j)
                bf[u][j] = buffer_load16(rb, kok ? (uint32_t)(((16 * j + (lane & 15)) * p.ldb + k) * 2) : kOffOutOfRange);
#pragma unroll
            for (int i = 0; i < MT; ++i)
                af[u][i] = buffer_load16(ra, kok ? (uint32_t)(((i * 16 + (lane & 15)) * p.lda + k) * 2) : kOffOutOfRange);
        }
    };
    auto mma_batch = [&]() {
#pragma unroll
        for (int u = 0; u < KU; ++u)
#pragma unroll
            for (int j = 0; j < 2; ++j)
#pragma unroll
                for (int i = 0; i < MT; ++i)
                    acc[j][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, af[u][i]),
                                                                        __builtin_bit_cast(bf16x8, bf[u][j]), acc[j][i],
                                                                        0, 0, 0);
    };
    load_batch(s0);
    // the slot-addressed epilogue operands go out behind the first batch of weights
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int t = 0; t < EPT; ++t)
        ein[t].load(p, em[t] < p.M ? em[t] : p.M - 1, en[t] < p.N ? en[t] : p.N - 1);
    __builtin_amdgcn_sched_barrier(0);
    mma_batch();
    for (int s = s0 + KU; s < s1; s += KU) {
        load_batch(s);
        mma_batch();
    }
    // lane l holds column l % 16 of block j and rows 4 (l / 16) + r of each 16-row tile
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int i = 0; i < MT; ++i)
#pragma unroll
            for (int r = 0; r < 4; ++r)
                red[wave][(i * 16 + 4 * (lane >> 4) + r) * NB + 16 * j + (lane & 15)] = acc[j][i][r];
    __syncthreads();
#pragma unroll
    for (int t = 0; t < EPT; ++t) {
        if (em[t] >= p.M || en[t] >= p.N) continue;
        const int e = threadIdx.x + t * NW * 64;
        float v = 0.0f;
#pragma unroll
        for (int w = 0; w < NW; ++w) v += red[w][e];
        if constexpr (EPI == kEpiStoreBf16) ((bf16*)p.C)[(int64_t)em[t] * p.ldc + en[t]] = (bf16)v;
        else if constexpr (EPI == kEpiStoreF32) ((float*)p.C)[(int64_t)em[t] * p.ldc + en[t]] = v;
        else ein[t].apply(p, em[t], en[t], v);
    }
}

// Streamed-weight variant for at most 16 rows, bf16 activations and K a multiple of 64
// (in_proj, x_proj and out_proj of a decode step). Loading MFMA fragments straight from
// global memory makes every load instruction touch 16 weight rows x 64 bytes (half cache
// lines of 16 rows), which streams at about half the rate of whole lines. Here every
// load instruction reads a block of 8 rows x 128 bytes (whole lines): a wave owns a
// contiguous run of up to NST 64-wide k stages and issues the loads of all of
// them (16 weight rows and the activation rows of each stage) at once, so its whole
// share is in flight after a single memory latency; registers hold it, since LDS could
// not. Each stage is then written to a small wave-private LDS buffer (XOR-swizzled rows)
// and read back as 16x16x32 MFMA fragments. The waves' partial tiles are summed through
// LDS at the end and go through the same epilogues.
constexpr int kGemvBK = 64;

__device__ __forceinline__ int gemv_swz(int row, int chunk) { return chunk ^ ((row >> 1) & 7); }

constexpr int kNormMaxK = 8192, kNormMaxMG = 256;  // norm prologue: K columns, rows x groups

template <int NW, int NST, int XB, int EPI, bool NORM = false>
__global__ __launch_bounds__(NW * 64) void gemm_gemv_kernel(SkinnyArgs p) {
    static_assert(NW >= 4, "one epilogue element per thread of the first 256");
    constexpr int SLOT = (2 + XB) * 1024;  // one stage: 16 weight rows, then 8 * XB activation rows, 128 B each
    __shared__ __attribute__((aligned(16))) char tr[NW][2][SLOT];
    __shared__ float red[NW][256];
    // norm prologue: norm_w over K and the per-(row, group) inverse RMS, staged once
    __shared__ __attribute__((aligned(16))) float nrm_w[NORM ? kNormMaxK : 4];
    __shared__ float nrm_inv[NORM ? kNormMaxMG : 1];
    const int n0 = blockIdx.x * 16;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;

    const int e = threadIdx.x;
    const int em = e >> 4, en = n0 + (e & 15);
    const bool ework = e < 256 && em < p.M && en < p.N;
    const int emc = em < p.M ? em : p.M - 1, enc = en < p.N ? en : p.N - 1;  // in-range for the fetch
    EpiIn<EPI> ein;
    ein.load_slot(p, emc);

    // this wave's stages [sb, sb + nst) of the K / 64 (nst <= NST, checked by the launcher)
    const int nall = p.K / kGemvBK;
    const int sb = wave * nall / NW, nst = (wave + 1) * nall / NW - sb;
    // lane l loads row l / 8 of a block, 16-byte chunk l % 8; weight rows past N and
    // activation rows past M lie outside the resources and read as zero
    const int lr = lane >> 3, lp = lane & 7;
    const __amdgpu_buffer_rsrc_t rb = buffer_rsrc(p.B + (int64_t)n0 * p.ldb, (uint32_t)(min(16, p.N - n0) * p.ldb * 2));
    const __amdgpu_buffer_rsrc_t ra = buffer_rsrc(p.A, (uint32_t)(p.M * p.lda * 2));
    const uint32_t k0b = (uint32_t)(sb * kGemvBK + lp * 8) * 2;
    const uint32_t wo0 = (uint32_t)(lr * p.ldb) * 2 + k0b, wo1 = (uint32_t)((8 + lr) * p.ldb) * 2 + k0b;
    // norm prologue operands go out first, so that waiting for them waits for nothing else
    constexpr int NSTG = NORM ? kNormMaxK / 4 / (NW * 64) : 1;
    float4 nwr[NSTG];
    float ssq = 0.0f;
    if constexpr (NORM) {
#pragma unroll
        for (int j = 0; j < NSTG; ++j) {
            const int i = threadIdx.x + j * NW * 64;
            nwr[j] = i < p.K / 4 ? ((const float4*)p.nrm_w)[i] : make_float4(0.f, 0.f, 0.f, 0.f);
        }
        if ((int)threadIdx.x < p.M * p.nrm_G) ssq = p.nrm_sumsq[threadIdx.x];
        __builtin_amdgcn_sched_barrier(0);
    }
    u32x4 w0[NST], w1[NST], xv[NST][XB];
#pragma unroll
    for (int st = 0; st < NST; ++st) {
        const bool ok = st < nst;
        w0[st] = buffer_load16(rb, ok ? wo0 + st * 128 : kOffOutOfRange);
        w1[st] = buffer_load16(rb, ok ? wo1 + st * 128 : kOffOutOfRange);
#pragma unroll
        for (int q = 0; q < XB; ++q)
            xv[st][q] = buffer_load16(ra, ok ? (uint32_t)((8 * q + lr) * p.lda) * 2 + k0b + st * 128 : kOffOutOfRange);
    }
    // the epilogue's slot-addressed operands go out behind the stream
    __builtin_amdgcn_sched_barrier(0);
    ein.load(p, emc, enc);
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (NORM) {
        // the same arithmetic as the separate norm kernel: 1 / sqrt(sumsq / gsize + eps),
        // then (g * inv) * norm_w rounded to bf16
#pragma unroll
        for (int j = 0; j < NSTG; ++j) {
            const int i = threadIdx.x + j * NW * 64;
            if (i < p.K / 4) *(float4*)&nrm_w[4 * i] = nwr[j];
        }
        if ((int)threadIdx.x < p.M * p.nrm_G) nrm_inv[threadIdx.x] = 1.0f / sqrtf(ssq / (float)p.nrm_gsize + p.nrm_eps);
        __syncthreads();
    }
    // the inverse RMS of this lane's activation rows (rows past M: 0) for one group per row
    auto inv_at = [&](int row, int k) { return row < p.M ? nrm_inv[row * p.nrm_G + (p.nrm_c0 + k) / p.nrm_gsize] : 0.0f; };
    float inv1[XB];
#pragma unroll
    for (int q = 0; q < XB; ++q) inv1[q] = NORM && 8 * q + lr < p.M ? nrm_inv[NORM ? (8 * q + lr) * p.nrm_G : 0] : 0.0f;

    // fragment rows: weights l % 16, activations l % (8 XB); chunk 4 j + l / 16 of substep j
    const int wr = lane & 15, xr = XB == 2 ? (lane & 15) : (lane & 7), cg = lane >> 4;
    f32x4 acc = f32x4{};
#pragma unroll
    for (int st = 0; st < NST; ++st) {
        if (st < nst) {
            char* t = tr[wave][st & 1];
            *(u32x4*)(t + lr * 128 + gemv_swz(lr, lp) * 16) = w0[st];
            *(u32x4*)(t + (8 + lr) * 128 + gemv_swz(8 + lr, lp) * 16) = w1[st];
#pragma unroll
            for (int q = 0; q < XB; ++q) {
                u32x4 xq = xv[st][q];
                if constexpr (NORM) {
                    const int k = (sb + st) * kGemvBK + lp * 8;
                    // one group per row (the usual case) needs no group index
                    const float inv = p.nrm_G == 1 ? inv1[q] : inv_at(8 * q + lr, k);
                    const float4 w0 = *(const float4*)&nrm_w[k], w1 = *(const float4*)&nrm_w[k + 4];
                    const float wv[8] = {w0.x, w0.y, w0.z, w0.w, w1.x, w1.y, w1.z, w1.w};
                    const bf16x8 x8 = __builtin_bit_cast(bf16x8, xq);
                    bf16x8 o;
#pragma unroll
                    for (int e = 0; e < 8; ++e) o[e] = (bf16)((float)x8[e] * inv * wv[e]);
                    xq = __builtin_bit_cast(u32x4, o);
                }
                *(u32x4*)(t + 2048 + (8 * q + lr) * 128 + gemv_swz(8 * q + lr, lp) * 16) = xq;
            }
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                const int c = 4 * j + cg;
                const bf16x8 wf = *(const bf16x8*)(t + wr * 128 + gemv_swz(wr, c) * 16);
                const bf16x8 xf = *(const bf16x8*)(t + 2048 + xr * 128 + gemv_swz(xr, c) * 16);
                acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xf, wf, acc, 0, 0, 0);
            }
        }
    }
    // lane l holds column l % 16 and rows 4 (l / 16) + r of the 16-row tile
#pragma unroll
    for (int r = 0; r < 4; ++r) red[wave][(4 * (lane >> 4) + r) * 16 + (lane & 15)] = acc[r];
    __syncthreads();
    if (!ework) return;
    float v = 0.0f;
#pragma unroll
    for (int w = 0; w < NW; ++w) v += red[w][e];
    if constexpr (EPI == kEpiStoreBf16) ((bf16*)p.C)[(int64_t)em * p.ldc + en] = (bf16)v;
    else if constexpr (EPI == kEpiStoreF32) ((float*)p.C)[(int64_t)em * p.ldc + en] = v;
    else ein.apply(p, em, en, v);
}

// waves per workgroup for the streamed variant (0: it does not apply). Grids that fill
// the CUs take 8 waves of up to 5 stages each (up to 10 for longer K; 4 waves for K up to
// 1280); small grids take 16 waves of up to 4 stages, so that the few CUs in use keep many
// blocks in flight. Shorter runs per wave shorten the tail after the loads land: with 8
// waves instead of 4 at K = 2560, the 2.8B half shard's decode in_proj+conv took 7.6
// instead of 8.4 us and its step 21.5 instead of 22.5 us (10 waves: 22.1 us).
// (Spreading N over exactly one workgroup per CU, ceil(N / 256) rows each, shortened the
// kernels' span but not a decode step, so the tiles stay 16 columns wide.)
int gemv_waves(const SkinnyArgs& p) {
    auto al16 = [](const void* q) { return ((uintptr_t)q & 15) == 0; };
    if (p.M > 16 || p.a_f32 || p.K % kGemvBK != 0 || p.lda % 8 != 0 || p.ldb % 8 != 0 || !al16(p.A) || !al16(p.B))
        return 0;
    if ((int64_t)p.M * p.lda * 2 >= (int64_t)1 << 31 || (int64_t)16 * p.ldb * 2 >= (int64_t)1 << 31) return 0;
    const int nall = p.K / kGemvBK;
    if ((p.N + 15) / 16 < 128) return nall <= 16 * 4 ? 16 : 0;
    if (nall <= 4 * 5) return 4;
    return nall <= 8 * 10 ? 8 : 0;
}

template <int EPI>
hipError_t launch_gemv(const SkinnyArgs& p, int nw, hipStream_t s) {
    const dim3 grid((unsigned)((p.N + 15) / 16)), block(nw * 64);
#define SSM_GEMV(NW, NST)                                                                  \
    if (p.M <= 8) SSM_LAUNCH((gemm_gemv_kernel<NW, NST, 1, EPI>), grid, block, 0, s, p);   \
    else SSM_LAUNCH((gemm_gemv_kernel<NW, NST, 2, EPI>), grid, block, 0, s, p);
    if (nw == 4) { SSM_GEMV(4, 5) }
    else if (nw == 8) { if (p.K / kGemvBK <= 8 * 5) { SSM_GEMV(8, 5) } else { SSM_GEMV(8, 10) } }
    else { SSM_GEMV(16, 4) }
#undef SSM_GEMV
    return hipGetLastError();
}

template <int MB, int NW, int KU, bool AF, int EPI>
void launch_one(const SkinnyArgs& p, dim3 grid, hipStream_t s) {
    SSM_LAUNCH((gemm_skinny_kernel<MB, NW, KU, AF, EPI>), grid, dim3(NW * 64), 0, s, p);
}

// 16-row tiles: each wave issues all of its k-steps at once when they fit in registers
template <int NW, bool AF, int EPI>
void launch_ku16(const SkinnyArgs& p, dim3 grid, int per, hipStream_t s) {
    if (per <= 2) launch_one<16, NW, 2, AF, EPI>(p, grid, s);
    else if (per <= 4) launch_one<16, NW, 4, AF, EPI>(p, grid, s);
    else if constexpr (AF) launch_one<16, NW, 8, AF, EPI>(p, grid, s);  // fp32 A takes twice the registers
    else if (per <= 8) launch_one<16, NW, 8, AF, EPI>(p, grid, s);
    else launch_one<16, NW, 12, AF, EPI>(p, grid, s);
}

template <int MB, bool AF, int EPI>
hipError_t launch_mb(const SkinnyArgs& p, hipStream_t s) {
    const dim3 grid((unsigned)((p.N + 15) / 16), (unsigned)((p.M + MB - 1) / MB));
    const int ksteps = (p.K + 31) / 32;
    if constexpr (MB == 16) {
        // many tiles: 8 waves, so two workgroups share a CU and every tile starts in the first
        // round; few tiles: 16 waves, so each wave's share of K stays short. (The state
        // epilogue keeps a state row per thread: at most 8 waves.)
        if constexpr (EPI == kEpiState) launch_ku16<8, AF, EPI>(p, grid, (ksteps + 7) / 8, s);
        else if ((int64_t)grid.x * grid.y < 128) launch_ku16<16, AF, EPI>(p, grid, (ksteps + 15) / 16, s);
        else launch_ku16<8, AF, EPI>(p, grid, (ksteps + 7) / 8, s);
    } else {
        // one thread per output element; enough waves that each streams at most 8 k-steps
        constexpr int KU = (MB <= 32 ? 6 : 4) / (AF ? 2 : 1);
        constexpr int NWMIN = MB * 16 / 64;
        constexpr int NWMAX = EPI == kEpiState ? 8 : 16;
        const int want = (ksteps + 7) / 8;
        if ((want > 8 || NWMIN > 8) && NWMAX >= 16) launch_one<MB, NWMAX, KU, AF, EPI>(p, grid, s);
        else launch_one<MB, (NWMIN > 8 ? NWMAX : 8), KU, AF, EPI>(p, grid, s);
    }
    return hipGetLastError();
}

template <bool AF, int EPI>
hipError_t launch_epi(const SkinnyArgs& p, hipStream_t s) {
    // narrow outputs (under 64 column tiles: x_proj) take 16-row tiles at any M, so that the
    // row tiles spread over more workgroups: at 64 rows x_proj 8.8 -> 4.5 us (1280-channel
    // shard) and 17.5 -> 7.8 us (3584-channel shard, K = 3584). The state step does so up to
    // 32 rows (32 sequences, 1280 channels: 7.0 -> 5.7 us; at 64 rows 16-row tiles were slower)
    if (p.M <= 16 || (EPI == kEpiState && p.M <= 32) || (EPI != kEpiState && (p.N + 15) / 16 < 64))
        return launch_mb<16, AF, EPI>(p, s);
    // the state epilogue holds a whole state row per thread: at most 32-row tiles (8 waves)
    if (p.M <= 32 || EPI == kEpiState) return launch_mb<32, AF, EPI>(p, s);
    if constexpr (EPI != kEpiState) return launch_mb<64, AF, EPI>(p, s);
    return hipErrorInvalidValue;
}

// Decode projections of more rows (bf16, K a multiple of 64): a workgroup owns a TM x TN
// output tile and its NW waves split K. Each wave streams its share of the tile's
// activation and weight rows into a ring of RD stages in its own part of LDS on the DMA
// path (buffer_load ... lds: whole lines, 8 rows x 128 bytes per instruction, no registers
// held), waits for them with its own vmcnt and reads them back as
// v_mfma_f32_16x16x32_bf16 fragments. No barrier sits inside the k loop, so each wave
// keeps RD - 1 stages in flight on its own. (A 64 x 64 tile kernel that moves both
// operands through a shared LDS ring with a barrier per 64-wide k-step fetched about 20
// bytes per clock per CU; the CUs take about 64 from L2. Staging the stages through
// registers instead lost most of the prefetch: the compiler's counter waits at the top of
// the k loop assumed few loads in flight.) The waves' partial tiles are summed through LDS;
// each thread then takes whole 8-column groups of the tile through the epilogue (plain
// stores, or the conv window of in_proj, 16-byte accesses throughout).
template <int TM, int TN, int NW, int RD, int EPI, int KC>
__global__ __launch_bounds__(NW * 64) void gemm_dtile_kernel(SkinnyArgs p) {
    constexpr int AB = TM / 8, BB = TN / 8;   // 8-row blocks of one stage
    constexpr int OPS = AB + BB;              // DMA instructions per stage
    constexpr int MT = TM / 16, NT = TN / 16;
    constexpr int SLOT = OPS * 1024;          // one stage: activation rows, then weight rows
    constexpr int RING = NW * RD * SLOT;
    constexpr int RED = NW * TM * TN * 4;
    constexpr int SMEM = RING > RED ? RING : RED;
    constexpr int G = TM * TN / 8 / (NW * 64);  // epilogue groups per thread
    static_assert(TM % 16 == 0 && TM <= 64 && TN % 16 == 0 && G >= 1 && G * NW * 64 * 8 == TM * TN, "tile");
    static_assert(RD >= 2 && (RD - 1) * OPS < 64, "stages in flight within the vmcnt range");
    __shared__ __attribute__((aligned(1024))) char smem[SMEM];
    // column tiles outer, row tiles inner: the row tiles of one column tile (which read
    // the same weight rows) take consecutive indices, hence one XCD's L2
    const int tiles_m = (p.M + TM - 1) / TM;
    const int t = xcd_contiguous((int)blockIdx.x, (int)gridDim.x);
    const int m0 = (t % tiles_m) * TM, n0 = (t / tiles_m) * TN;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;

    // epilogue group k of this thread: tile row er[k], columns ec[k] .. ec[k] + 7
    int er[G], ec[G], slot[G];
#pragma unroll
    for (int k = 0; k < G; ++k) {
        const int g = threadIdx.x + k * NW * 64;
        er[k] = g / (TN / 8);
        ec[k] = (g % (TN / 8)) * 8;
        slot[k] = 0;
        if constexpr (EPI == kEpiConv) slot[k] = p.slot[min(m0 + er[k], p.M - 1)];
    }
    // the conv window operands of the epilogue groups (conv width KC) go out before the
    // weight stream, so they arrive with its first stage instead of after its last. (The
    // compiler waits for the slot indices with a full vector-memory count, which must
    // happen before any stage is in flight.)
    constexpr int KW = EPI == kEpiConv ? KC : 2;
    ConvWindow8<bf16, KW> cw[G];
    bool inconv[G];
#pragma unroll
    for (int k = 0; k < G; ++k) {
        const int m = m0 + er[k], c = n0 + ec[k] - p.conv_lo;
        inconv[k] = EPI == kEpiConv && m < p.M && c >= 0 && c < p.conv_n;
        if (inconv[k]) {
            const int sc = slot_ok(slot[k], p.S) ? slot[k] : 0;
            cw[k].load((const bf16*)p.conv_pool + ((int64_t)sc * p.conv_n + c) * (KW - 1),
                       (const bf16*)p.conv_w + (int64_t)c * KW, (const bf16*)p.conv_b + c);
        }
    }
    __builtin_amdgcn_sched_barrier(0);

    const int nall = p.K / kGemvBK;
    const int sb = wave * nall / NW, nst = (wave + 1) * nall / NW - sb;
    // lane l of a DMA instruction lands at byte 16 l of its 1 KB block: row l / 8, stored
    // chunk l % 8, which holds the row's chunk (l % 8) ^ ((row >> 1) & 7) (the swizzle the
    // fragment reads undo). Rows past M or N lie outside the resources and land as zero.
    const int lr = lane >> 3, lp = lane & 7;
    const __amdgpu_buffer_rsrc_t ra =
        buffer_rsrc((const bf16*)p.A + (int64_t)m0 * p.lda, (uint32_t)(min(TM, p.M - m0) * p.lda * 2));
    const __amdgpu_buffer_rsrc_t rb = buffer_rsrc(p.B + (int64_t)n0 * p.ldb, (uint32_t)(min(TN, p.N - n0) * p.ldb * 2));
    uint32_t aoff[AB], boff[BB];
#pragma unroll
    for (int q = 0; q < AB; ++q) {
        const int r = 8 * q + lr;
        aoff[q] = (uint32_t)(r * p.lda) * 2 + (uint32_t)(gemv_swz(r, lp) * 16 + sb * kGemvBK * 2);
    }
#pragma unroll
    for (int q = 0; q < BB; ++q) {
        const int r = 8 * q + lr;
        boff[q] = (uint32_t)(r * p.ldb) * 2 + (uint32_t)(gemv_swz(r, lp) * 16 + sb * kGemvBK * 2);
    }
    const uint32_t ring = (uint32_t)(uintptr_t)(lds_ptr_t)(smem + wave * RD * SLOT);
    // stage st of this wave's run into ring slot j; stages past the run read out of range
    // (no memory touched), so every refill is OPS instructions and the counter waits are exact
    auto stage_dma = [&](int st, int j) {
        const bool ok = st < nst;
        const uint32_t soff = __builtin_amdgcn_readfirstlane(ok ? (uint32_t)st * kGemvBK * 2 : 0u);  // wave-uniform
        const uint32_t base = ring + (uint32_t)(j * SLOT);
#pragma unroll
        for (int q = 0; q < AB; ++q)
            dma16(ra, ok ? aoff[q] : kOffOutOfRange, soff, __builtin_amdgcn_readfirstlane(base + q * 1024));
#pragma unroll
        for (int q = 0; q < BB; ++q)
            dma16(rb, ok ? boff[q] : kOffOutOfRange, soff, __builtin_amdgcn_readfirstlane(base + (AB + q) * 1024));
    };
#pragma unroll
    for (int j = 0; j < RD; ++j) stage_dma(j, j);

    const int fr = lane & 15, cg = lane >> 4;
    f32x4 acc[MT][NT];
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int jn = 0; jn < NT; ++jn) acc[i][jn] = f32x4{};
    for (int st = 0; st < nst; ++st) {
        const int j = st % RD;
        wait_vm<(RD - 1) * OPS>();  // stage st has landed; the RD - 1 after it may not have
        const char* abuf = smem + (wave * RD + j) * SLOT;
        const char* wbuf = abuf + AB * 1024;
        // the whole stage goes to registers first and its slot is refilled before the
        // MFMAs, so RD stages (not RD - 1) are in flight while the wave multiplies
        bf16x8 af[2][MT], wf[2][NT];
#pragma unroll
        for (int s = 0; s < 2; ++s) {
            const int c = 4 * s + cg;
#pragma unroll
            for (int i = 0; i < MT; ++i)
                af[s][i] = *(const bf16x8*)(abuf + (16 * i + fr) * 128 + gemv_swz(16 * i + fr, c) * 16);
#pragma unroll
            for (int jn = 0; jn < NT; ++jn)
                wf[s][jn] = *(const bf16x8*)(wbuf + (16 * jn + fr) * 128 + gemv_swz(16 * jn + fr, c) * 16);
        }
        wait_lgkm0();  // the slot's fragments are read before it is refilled
        stage_dma(st + RD, j);
        __builtin_amdgcn_sched_barrier(0);  // no MFMA moves above the refill
#pragma unroll
        for (int s = 0; s < 2; ++s)
#pragma unroll
            for (int jn = 0; jn < NT; ++jn)
#pragma unroll
                for (int i = 0; i < MT; ++i)
                    acc[i][jn] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[s][i], wf[s][jn], acc[i][jn], 0, 0, 0);
    }
    wait_vm<0>();  // every DMA (the out-of-range refills too) has landed before LDS is reused
    // lane l holds column 16 jn + l % 16, rows 16 i + 4 (l / 16) + r of the tile
    __syncthreads();
    float* red = (float*)smem;
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int jn = 0; jn < NT; ++jn)
#pragma unroll
            for (int r = 0; r < 4; ++r) red[(wave * TM + 16 * i + 4 * cg + r) * TN + 16 * jn + fr] = acc[i][jn][r];
    __syncthreads();
#pragma unroll
    for (int k = 0; k < G; ++k) {
        const int m = m0 + er[k], n = n0 + ec[k];
        float v[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = 0.0f;
#pragma unroll
        for (int w = 0; w < NW; ++w) {
            const float* q = red + (w * TM + er[k]) * TN + ec[k];
            const float4 a = *(const float4*)q, b = *(const float4*)(q + 4);
            v[0] += a.x; v[1] += a.y; v[2] += a.z; v[3] += a.w; v[4] += b.x; v[5] += b.y; v[6] += b.z; v[7] += b.w;
        }
        if (m >= p.M || n >= p.N) continue;
        if constexpr (EPI == kEpiStoreF32) {
            float* o = (float*)p.C + (int64_t)m * p.ldc + n;
            *(float4*)o = make_float4(v[0], v[1], v[2], v[3]);
            *(float4*)(o + 4) = make_float4(v[4], v[5], v[6], v[7]);
        } else {
            bf16x8 o;
#pragma unroll
            for (int e = 0; e < 8; ++e) o[e] = (bf16)v[e];
            const int c = n - p.conv_lo;
            if (!inconv[k]) {
                *(bf16x8*)((bf16*)p.C + (int64_t)m * p.ldc + n) = o;
                continue;
            }
            if constexpr (EPI == kEpiConv) {
                // the stored (rounded) projection outputs enter the window
                float cur[8], out[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) cur[e] = (float)o[e];
                const bool ok = slot_ok(slot[k], p.S);
                cw[k].step(cur, (bf16*)p.conv_pool + ((int64_t)slot[k] * p.conv_n + c) * (KW - 1), ok, out);
                if (!ok) atomicOr(p.status, SSM_STATUS_BAD_SLOT);
                bf16x8 uo;
#pragma unroll
                for (int e = 0; e < 8; ++e) uo[e] = (bf16)out[e];
                *(bf16x8*)((bf16*)p.u + (int64_t)m * p.conv_n + c) = uo;
            }
        }
    }
}

// the tile kernel's shapes: bf16 activations, K a multiple of 64, whole 8-column groups
// (N, the row strides and the conv column range multiples of 8), 16-byte aligned operands
bool dtile_fits(const SkinnyArgs& p, int epi) {
    auto al16 = [](const void* q) { return ((uintptr_t)q & 15) == 0; };
    if (p.a_f32 || p.K % kGemvBK != 0 || p.N % 8 != 0 || p.lda % 8 != 0 || p.ldb % 8 != 0 || p.ldc % 8 != 0 ||
        !al16(p.A) || !al16(p.B) || !al16(p.C))
        return false;
    if ((int64_t)64 * p.lda * 2 >= (int64_t)1 << 31 || (int64_t)64 * p.ldb * 2 >= (int64_t)1 << 31) return false;
    if (epi == kEpiConv && (p.conv_lo % 8 != 0 || p.conv_n % 8 != 0 || p.Kc < 2 || p.Kc > 4 || !al16(p.u) ||
                            !al16(p.conv_w) || !al16(p.conv_b) || !al16(p.conv_pool)))
        return false;
    return true;
}

template <int TM, int TN, int NW, int RD, int EPI>
hipError_t launch_dtile(const SkinnyArgs& p, hipStream_t s) {
    const dim3 grid((unsigned)(((p.M + TM - 1) / TM) * ((p.N + TN - 1) / TN))), block(NW * 64);
    if constexpr (EPI == kEpiConv) {
        switch (p.Kc) {
            case 2: SSM_LAUNCH((gemm_dtile_kernel<TM, TN, NW, RD, EPI, 2>), grid, block, 0, s, p); break;
            case 3: SSM_LAUNCH((gemm_dtile_kernel<TM, TN, NW, RD, EPI, 3>), grid, block, 0, s, p); break;
            default: SSM_LAUNCH((gemm_dtile_kernel<TM, TN, NW, RD, EPI, 4>), grid, block, 0, s, p); break;
        }
    } else {
        SSM_LAUNCH((gemm_dtile_kernel<TM, TN, NW, RD, EPI, 0>), grid, block, 0, s, p);
    }
    return hipGetLastError();
}

// 17..512 rows over outputs of at least 128 tiles: 64 x 64 tiles above 128 rows when they
// give 128 workgroups, else 64 x 32 tiles (both 4 waves, one stage in flight per wave while
// the other is multiplied), else 32 x 32 tiles of 2 waves with 3 stages in flight. Measured
// with the weights coming from the MALL (rotated over copies, as in a decode step):
// in_proj + conv window of the 2.8B quarter shard (2560 x 2560) at 256 rows 14.0 us (17.8
// for 64 x 64 DMA tiles in two K-slices plus the conv kernel that added them) and at 128
// rows 10.0 us; its out_proj (2560 x 1280) 7.7 and 5.8 us (8.9 and 15.3 on 64 x 64 DMA
// tiles); the hybrid shard's in_proj + conv (7168 x 3584) at 64 rows 13.5 us (23.8 with L2-warm
// weights on the 32-column kernel) and its out_proj (3584 x 3584) 9.5 us (17.9 on 16-column
// tiles). hipErrorNotSupported when it does not apply.
template <int EPI>
hipError_t launch_dtile_pick(const SkinnyArgs& p, hipStream_t s) {
    if (p.M <= 16 || p.M > 512 || !dtile_fits(p, EPI)) return hipErrorNotSupported;
    const int64_t tm64 = (p.M + 63) / 64, tm32 = (p.M + 31) / 32, tn64 = (p.N + 63) / 64, tn32 = (p.N + 31) / 32;
    if (p.M > 128 && tm64 * tn64 >= 128) return launch_dtile<64, 64, 4, 2, EPI>(p, s);
    if (tm64 * tn32 >= 128) return launch_dtile<64, 32, 4, 2, EPI>(p, s);
    if (tm32 * tn32 >= 128) return launch_dtile<32, 32, 2, 4, EPI>(p, s);
    return hipErrorNotSupported;
}

// 32-column tiles for 17..64 bf16 rows when they still give at least 192 workgroups.
// Measured at 64 rows: the 7168-wide in_proj (224 workgroups) 36.6 -> 24.3 us; with 80 or
// 112 workgroups (2560 or 3584 columns) the 16-column tiles were faster.
bool use_skinny32(const SkinnyArgs& p) {
    return !p.a_f32 && p.M > 16 && p.M <= 64 && (p.N + 31) / 32 >= 192 && p.K % 8 == 0 && p.lda % 8 == 0 &&
           p.ldb % 8 == 0;
}

template <int EPI>
hipError_t launch_skinny32(const SkinnyArgs& p, hipStream_t s) {
    const int ksteps = (p.K + 31) / 32;
    if (p.M <= 32) {
        const dim3 grid((unsigned)((p.N + 31) / 32), 1);
        if ((ksteps + 15) / 16 <= 2) SSM_LAUNCH((gemm_skinny32_kernel<32, 16, 2, EPI>), grid, dim3(1024), 0, s, p);
        else SSM_LAUNCH((gemm_skinny32_kernel<32, 16, 4, EPI>), grid, dim3(1024), 0, s, p);
    } else {
        const dim3 grid((unsigned)((p.N + 31) / 32), 1);
        if ((ksteps + 7) / 8 <= 2) SSM_LAUNCH((gemm_skinny32_kernel<64, 8, 2, EPI>), grid, dim3(512), 0, s, p);
        else SSM_LAUNCH((gemm_skinny32_kernel<64, 8, 4, EPI>), grid, dim3(512), 0, s, p);
    }
    return hipGetLastError();
}

// Float32 operands, at most 64 rows (the decode projections of a float32 layer): the
// weight stream is 4 bytes per element, so moving it in whole cache lines matters as much as
// in the bf16 kernel above. A workgroup owns CT tiles of 16 output columns; its NW waves
// split K into runs of 32-wide stages (128 bytes of a float32 row). Each stage arrives by
// whole-line loads, 8 rows x 128 bytes per instruction (16 CT weight rows, then the 8 XB
// activation rows), NST stages ahead in registers; it is written to a wave-private LDS buffer
// (XOR-swizzled 16-byte chunks) and read back as v_mfma_f32_16x16x4_f32 operands: lane l
// takes the float4 of chunk 4 j + l / 16 of row l % 16, and MFMA t of group j uses
// component t, so operand and weight agree on every k. Rows past M or N read as zero. The
// waves' partial tiles are summed through the same LDS at the end.
constexpr int kF32Stage = 32;  // k per stage: one 128-byte line of a float32 row

// CONV: the conv window in the epilogue (launch_gemv_f32_conv). A thread's epilogue items are
// e = tid + i NW 64; their slot indices go out before the weight stream and the
// slot-addressed window inputs, taps and bias right after it, so they land with the stream.
template <int ROLE, int NW, int NST, int XB, int CT = 1, bool CONV = false>
__global__ __launch_bounds__(NW * 64) void gemv_f32_stream_kernel(int M, int N, int K, const float* __restrict__ A,
                                                                  int64_t lda, const float* __restrict__ B,
                                                                  int64_t ldb, float* __restrict__ C, int64_t ldc,
                                                                  F32ConvEpi cv = {}) {
    constexpr int WR = 16 * CT;                // weight rows of a workgroup (CT 16-column tiles)
    constexpr int ROWS = WR + 8 * XB;          // LDS rows of one stage: weights, then activations
    constexpr int MT = (8 * XB + 15) / 16;     // 16-row output tiles
    constexpr int WBUF = ROWS * 128;           // bytes of a wave's buffer
    static_assert(WBUF >= CT * MT * 16 * 16 * 4, "the partial tiles fit the wave's buffer");
    constexpr int NE = CT * MT * 256;          // epilogue items: (tile, row, column)
    constexpr int EL = (NE + NW * 64 - 1) / (NW * 64);
    __shared__ __attribute__((aligned(16))) char tr[NW][WBUF];
    const int n0 = blockIdx.x * WR;
    // row tiles of 8 XB activation rows along blockIdx.y (one tile when the grid has one row)
    const int m0 = blockIdx.y * 8 * XB;
    A += (int64_t)m0 * lda;
    C += (int64_t)m0 * ldc;
    M = min(M - m0, 8 * XB);
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    // epilogue item i of this thread: its row, column, and (CONV) slot
    auto item = [&](int i, int& m, int& n) {
        const int e = (int)threadIdx.x + i * NW * 64;
        m = (e / 16) % (MT * 16);
        n = n0 + 16 * (e / (MT * 256)) + (e & 15);
        return e < NE && m < M && n < N;
    };
    int eslot[CONV ? EL : 1];
    if constexpr (CONV) {
#pragma unroll
        for (int i = 0; i < EL; ++i) {
            int m, n;
            eslot[i] = item(i, m, n) ? cv.slot[m0 + m] : 0;
        }
    }
    const int nall = K / kF32Stage;
    const int sb = wave * nall / NW, nst = (wave + 1) * nall / NW - sb;
    const int lr = lane >> 3, lp = lane & 7;
    const __amdgpu_buffer_rsrc_t rb = buffer_rsrc(B + (int64_t)n0 * ldb, (uint32_t)(min(WR, N - n0) * ldb * 4));
    const __amdgpu_buffer_rsrc_t ra = buffer_rsrc(A, (uint32_t)(M * lda * 4));
    const uint32_t kb = (uint32_t)(sb * kF32Stage + lp * 4) * 4;
    uint32_t wo[2 * CT], xo[XB];
#pragma unroll
    for (int q = 0; q < 2 * CT; ++q) wo[q] = (uint32_t)((8 * q + lr) * ldb) * 4 + kb;
#pragma unroll
    for (int q = 0; q < XB; ++q) xo[q] = (uint32_t)((8 * q + lr) * lda) * 4 + kb;

    u32x4 wv[NST][2 * CT], xv[NST][XB];
    auto issue = [&](int j, int st) {  // stage st of this wave's run into register slot j
        const bool ok = st < nst;
#pragma unroll
        for (int q = 0; q < 2 * CT; ++q) wv[j][q] = buffer_load16(rb, ok ? wo[q] + st * 128 : kOffOutOfRange);
#pragma unroll
        for (int q = 0; q < XB; ++q) xv[j][q] = buffer_load16(ra, ok ? xo[q] + st * 128 : kOffOutOfRange);
    };
#pragma unroll
    for (int j = 0; j < NST; ++j) issue(j, j);
    // (CONV) each item's window: K - 1 cached inputs, K taps, bias (channel 0 for columns
    // outside the conv path and slot 0 for a bad slot: read, never used)
    float ehv[CONV ? EL : 1][kMaxConv - 1], ewv[CONV ? EL : 1][kMaxConv], ebv[CONV ? EL : 1];
    if constexpr (CONV) {
        const int Kc = cv.K;
#pragma unroll
        for (int i = 0; i < EL; ++i) {
            int m, n;
            item(i, m, n);
            const int c = n < cv.conv_n ? n : 0;
            const int sc = eslot[i] >= 0 && eslot[i] < cv.S ? eslot[i] : 0;
            const float* hist = cv.conv_pool + ((int64_t)sc * cv.conv_n + c) * (Kc - 1);
#pragma unroll
            for (int j = 0; j < kMaxConv - 1; ++j) ehv[i][j] = hist[j < Kc - 1 ? j : Kc - 2];
#pragma unroll
            for (int j = 0; j < kMaxConv; ++j) ewv[i][j] = cv.w[(int64_t)c * Kc + (j < Kc ? j : Kc - 1)];
            ebv[i] = cv.b[c];
        }
    }

    char* t = tr[wave];
    const int wr = lane & 15, cg = lane >> 4;
    f32x4 acc[CT][MT];
#pragma unroll
    for (int ct = 0; ct < CT; ++ct)
#pragma unroll
        for (int i = 0; i < MT; ++i) acc[ct][i] = f32x4{};
    for (int base = 0; base < nst; base += NST) {
#pragma unroll
        for (int j = 0; j < NST; ++j) {
            if (base + j < nst) {
#pragma unroll
                for (int q = 0; q < 2 * CT; ++q)
                    *(u32x4*)(t + (8 * q + lr) * 128 + gemv_swz(8 * q + lr, lp) * 16) = wv[j][q];
#pragma unroll
                for (int q = 0; q < XB; ++q)
                    *(u32x4*)(t + (WR + 8 * q + lr) * 128 + gemv_swz(WR + 8 * q + lr, lp) * 16) = xv[j][q];
                issue(j, base + j + NST);  // refill the slot just written out
#pragma unroll
                for (int g = 0; g < 2; ++g) {
                    const int c = 4 * g + cg;
                    f32x4 xf[MT];
#pragma unroll
                    for (int i = 0; i < MT; ++i) {
                        // rows past the staged 8 XB activation rows repeat earlier ones; their
                        // outputs lie past M and are never stored
                        const int ar = WR + ((16 * i + wr) % (8 * XB));
                        xf[i] = *(const f32x4*)(t + ar * 128 + gemv_swz(ar, c) * 16);
                    }
#pragma unroll
                    for (int ct = 0; ct < CT; ++ct) {
                        const int rw = 16 * ct + wr;
                        const f32x4 wf = *(const f32x4*)(t + rw * 128 + gemv_swz(rw, c) * 16);
#pragma unroll
                        for (int i = 0; i < MT; ++i)
#pragma unroll
                            for (int u = 0; u < 4; ++u)
                                acc[ct][i] = __builtin_amdgcn_mfma_f32_16x16x4f32(xf[i][u], wf[u], acc[ct][i], 0, 0, 0);
                    }
                }
            }
        }
    }
    // lane l holds column l % 16 and rows 16 i + 4 (l / 16) + r of tile (ct, i)
    __syncthreads();
    float* red = (float*)t;
#pragma unroll
    for (int ct = 0; ct < CT; ++ct)
#pragma unroll
        for (int i = 0; i < MT; ++i)
#pragma unroll
            for (int r = 0; r < 4; ++r) red[((ct * MT + i) * 16 + 4 * cg + r) * 16 + wr] = acc[ct][i][r];
    __syncthreads();
#pragma unroll
    for (int i = 0; i < EL; ++i) {
        int m, n;
        if (!item(i, m, n)) continue;
        const int e = (int)threadIdx.x + i * NW * 64;
        float v = 0.0f;
#pragma unroll
        for (int w = 0; w < NW; ++w) v += ((const float*)tr[w])[e];
        if constexpr (CONV) {
            if (n < cv.conv_n) {
                // the conv window step of the conv kernel: bias, the cached inputs, then this
                // token's input; SiLU; the window shifts by one
                const int Kc = cv.K, slot = eslot[i];
                float* u = cv.u + (int64_t)(m0 + m) * cv.conv_n + n;
                if (slot < 0 || slot >= cv.S) {
                    atomicOr(cv.status, SSM_STATUS_BAD_SLOT);
                    *u = 0.0f;
                    continue;
                }
                float acc = ebv[i];
#pragma unroll
                for (int j = 0; j < kMaxConv - 1; ++j)
                    if (j < Kc - 1) acc += ewv[i][j] * ehv[i][j];
                float wl = 0.0f;
#pragma unroll
                for (int j = 0; j < kMaxConv; ++j)
                    if (j == Kc - 1) wl = ewv[i][j];
                acc += wl * v;
                *u = silu_f(acc);
                float* hist = cv.conv_pool + ((int64_t)slot * cv.conv_n + n) * (Kc - 1);
#pragma unroll
                for (int j = 0; j < kMaxConv - 2; ++j)
                    if (j < Kc - 2) hist[j] = ehv[i][j + 1];
                hist[Kc - 2] = v;
                continue;
            }
        }
        C[(int64_t)m * ldc + n] = v;
    }
}

template <int ROLE, int NW, bool CONV = false>
hipError_t launch_f32_stream_nw(int M, int N, int K, const float* A, int64_t lda, const float* B, int64_t ldb,
                                float* C, int64_t ldc, hipStream_t s, const F32ConvEpi& cv = {}) {
    const dim3 grid((unsigned)((N + 15) / 16)), block(NW * 64);
    // 33..64 rows over wide outputs: two 16-column tiles per workgroup, so each staged block
    // of activation rows serves 32 columns (half the activation re-reads; the hybrid shard's
    // float32 in_proj of 64 rows 29.8 -> 28.5 us, where its 3.3 GFLOP take 21 us at the fp32
    // MFMA peak)
    if constexpr (NW == 8) {
        if (M > 32 && M <= 64 && (N + 31) / 32 >= 128) {
            const dim3 g2((unsigned)((N + 31) / 32));
            if (M <= 48) SSM_LAUNCH((gemv_f32_stream_kernel<ROLE, NW, 2, 6, 2, CONV>), g2, block, 0, s, M, N, K, A, lda, B, ldb, C, ldc, cv);
            else SSM_LAUNCH((gemv_f32_stream_kernel<ROLE, NW, 2, 8, 2, CONV>), g2, block, 0, s, M, N, K, A, lda, B, ldb, C, ldc, cv);
            return hipGetLastError();
        }
    }
#define SSM_F32S(XB, NST) \
    SSM_LAUNCH((gemv_f32_stream_kernel<ROLE, NW, NST, XB, 1, CONV>), grid, block, 0, s, M, N, K, A, lda, B, ldb, C, ldc, cv)
    if (M <= 8) SSM_F32S(1, 3);
    else if (M <= 16) SSM_F32S(2, 3);
    else if (M <= 32) SSM_F32S(4, 3);
    else if constexpr (NW <= 8) {
        if (M <= 48) SSM_F32S(6, 2);
        else SSM_F32S(8, 2);   // 64 activation rows: 10 KB of LDS per wave
    }
    else return hipErrorNotSupported;
#undef SSM_F32S
    return hipGetLastError();
}

template <int ROLE, bool CONV = false>
hipError_t launch_f32_stream_role(int M, int N, int K, const float* A, int64_t lda, const float* B, int64_t ldb,
                                  float* C, int64_t ldc, hipStream_t s, const F32ConvEpi& cv = {}) {
    // few column tiles (x_proj: 16): 16 waves, so that each wave's run of K stays short; more
    // than 8 rows are cut into 8-row tiles along the grid's second dimension, so that more
    // CUs share the stream and each reads 8 activation rows instead of all of them (the
    // hybrid shard's x_proj of 64 rows: 16 workgroups each reading all 64 rows took 14 us,
    // 64 of 16-row tiles 9.1 us, 128 of 8-row tiles 8.1 us)
    if ((N + 15) / 16 < 128) {
        if (M <= 8) return launch_f32_stream_nw<ROLE, 16, CONV>(M, N, K, A, lda, B, ldb, C, ldc, s, cv);
        const dim3 grid((unsigned)((N + 15) / 16), (unsigned)((M + 7) / 8)), block(16 * 64);
        SSM_LAUNCH((gemv_f32_stream_kernel<ROLE, 16, 3, 1, 1, CONV>), grid, block, 0, s, M, N, K, A, lda, B, ldb, C, ldc, cv);
        return hipGetLastError();
    }
    return launch_f32_stream_nw<ROLE, 8, CONV>(M, N, K, A, lda, B, ldb, C, ldc, s, cv);
}

}  // namespace

hipError_t launch_gemv_norm(const SkinnyArgs& p, hipStream_t s) {
    if (p.M <= 0 || p.N <= 0) return hipSuccess;
    const int nw = gemv_waves(p);
    // grids that fill the CUs only (4 or 8 waves): the 16-wave small-grid variant has no LDS
    // left for the staged norm weights
    if ((nw != 4 && nw != 8) || p.K > kNormMaxK || p.M * p.nrm_G > kNormMaxMG || p.nrm_gsize <= 0 ||
        p.nrm_gsize % 8 != 0 || ((uintptr_t)p.nrm_w & 15) != 0)
        return hipErrorNotSupported;
    const dim3 grid((unsigned)((p.N + 15) / 16)), block(nw * 64);
#define SSM_GEMV_N(NW, NST)                                                                              \
    if (p.M <= 8) SSM_LAUNCH((gemm_gemv_kernel<NW, NST, 1, kEpiStoreBf16, true>), grid, block, 0, s, p);   \
    else SSM_LAUNCH((gemm_gemv_kernel<NW, NST, 2, kEpiStoreBf16, true>), grid, block, 0, s, p);
    if (nw == 4) { SSM_GEMV_N(4, 5) }
    else if (p.K / kGemvBK <= 8 * 5) { SSM_GEMV_N(8, 5) }
    else { SSM_GEMV_N(8, 10) }
#undef SSM_GEMV_N
    return hipGetLastError();
}

hipError_t launch_gemm_skinny(const SkinnyArgs& p, SkinnyEpi epi, hipStream_t s) {
    if (p.M <= 0 || p.N <= 0) return hipSuccess;
    if (epi == kSkinnyStoreBf16 || epi == kSkinnyConv) {
        const hipError_t e = epi == kSkinnyConv ? launch_dtile_pick<kEpiConv>(p, s) : launch_dtile_pick<kEpiStoreBf16>(p, s);
        if (e != hipErrorNotSupported) return e;
    }
    if (use_skinny32(p)) {
        switch (epi) {
            case kSkinnyStoreBf16: return launch_skinny32<kEpiStoreBf16>(p, s);
            case kSkinnyStoreF32: return launch_skinny32<kEpiStoreF32>(p, s);
            case kSkinnyConv: return launch_skinny32<kEpiConv>(p, s);
            default: break;
        }
    }
    if (const int nw = gemv_waves(p)) {
        switch (epi) {
            case kSkinnyStoreBf16: return launch_gemv<kEpiStoreBf16>(p, nw, s);
            case kSkinnyStoreF32: return launch_gemv<kEpiStoreF32>(p, nw, s);
            case kSkinnyConv: return launch_gemv<kEpiConv>(p, nw, s);
            default: break;
        }
    }
    switch (epi) {
        case kSkinnyStoreBf16: return p.a_f32 ? launch_epi<true, kEpiStoreBf16>(p, s) : launch_epi<false, kEpiStoreBf16>(p, s);
        case kSkinnyStoreF32: return p.a_f32 ? launch_epi<true, kEpiStoreF32>(p, s) : launch_epi<false, kEpiStoreF32>(p, s);
        case kSkinnyConv: return launch_epi<false, kEpiConv>(p, s);
        case kSkinnyState: return launch_epi<true, kEpiState>(p, s);
    }
    return hipErrorInvalidValue;
}

}  // namespace ssm


namespace ssm {

namespace {
bool f32_stream_fits(int64_t M, int64_t K, const float* A, int64_t lda, const float* B, int64_t ldb) {
    auto al16 = [](const void* q) { return ((uintptr_t)q & 15) == 0; };
    return M <= 64 && K % kF32Stage == 0 && lda % 4 == 0 && ldb % 4 == 0 && al16(A) && al16(B) &&
           M * lda * 4 < ((int64_t)1 << 31) && 16 * ldb * 4 < ((int64_t)1 << 31);
}
}  // namespace

bool gemv_f32_conv_fits(int64_t M, int64_t N, int64_t K, const float* A, int64_t lda, const float* B, int64_t ldb,
                        const F32ConvEpi& cv) {
    return f32_stream_fits(M, K, A, lda, B, ldb) && cv.K >= 2 && cv.K <= kMaxConv && cv.conv_n <= N;
}

hipError_t launch_gemv_f32_conv(int64_t M, int64_t N, int64_t K, const float* A, int64_t lda, const float* B,
                                int64_t ldb, float* C, int64_t ldc, const F32ConvEpi& cv, hipStream_t s) {
    if (M <= 0 || N <= 0) return hipSuccess;
    if (!gemv_f32_conv_fits(M, N, K, A, lda, B, ldb, cv)) return hipErrorNotSupported;
    return launch_f32_stream_role<kGemmInProj, true>((int)M, (int)N, (int)K, A, lda, B, ldb, C, ldc, s, cv);
}

hipError_t launch_gemv_f32_stream(int role, int64_t M, int64_t N, int64_t K, const float* A, int64_t lda,
                                  const float* B, int64_t ldb, float* C, int64_t ldc, hipStream_t s) {
    if (M <= 0 || N <= 0) return hipSuccess;
    if (!f32_stream_fits(M, K, A, lda, B, ldb)) return hipErrorNotSupported;
    const int m = (int)M, n = (int)N, k = (int)K;
    switch (role) {
        case kGemmInProj: return launch_f32_stream_role<kGemmInProj>(m, n, k, A, lda, B, ldb, C, ldc, s);
        case kGemmXProj: return launch_f32_stream_role<kGemmXProj>(m, n, k, A, lda, B, ldb, C, ldc, s);
        case kGemmDtProj: return launch_f32_stream_role<kGemmDtProj>(m, n, k, A, lda, B, ldb, C, ldc, s);
        case kGemmOutProj: return launch_f32_stream_role<kGemmOutProj>(m, n, k, A, lda, B, ldb, C, ldc, s);
        default: return launch_f32_stream_role<kGemmGeneric>(m, n, k, A, lda, B, ldb, C, ldc, s);
    }
}

}  // namespace ssm
