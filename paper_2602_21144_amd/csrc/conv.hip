// Causal depthwise conv1d + SiLU of the SSM path (Section IV-B: Conv1d with groups equal
// to the channel count, so it runs on the shard's own channels with no communication),
// and the convolution half of the SSM cache (Section IV-A).
//
// u[t][c] = SiLU(b[c] + sum_j w[c][j] * xt[t - (K-1) + j][c]) over the packed batch, where
// positions before a sequence's first token come from its cached history (oldest
// first) when it continues, else are zero. Each thread owns 8 consecutive channels and
// a run of tokens, sliding its K-tap window in registers: every input row is read once
// per run (plus K-1 rows of overlap), with 16-byte loads and stores.
#include "common.h"

namespace ssm {
namespace {

constexpr int kCV = 8;   // channels per thread
constexpr int kTT = 8;   // tokens per thread (prefill)

template <typename T> struct Vec8;
template <> struct Vec8<bf16> {
    static __device__ __forceinline__ void load(const bf16* p, float* o) {
        bf16x8 v = *(const bf16x8*)p;
#pragma unroll
        for (int i = 0; i < 8; ++i) o[i] = (float)v[i];
    }
    static __device__ __forceinline__ void store(bf16* p, const float* o) {
        bf16x8 v;
#pragma unroll
        for (int i = 0; i < 8; ++i) v[i] = (bf16)o[i];
        *(bf16x8*)p = v;
    }
};
template <> struct Vec8<float> {
    static __device__ __forceinline__ void load(const float* p, float* o) {
        float4 a = *(const float4*)p, b = *(const float4*)(p + 4);
        o[0] = a.x; o[1] = a.y; o[2] = a.z; o[3] = a.w; o[4] = b.x; o[5] = b.y; o[6] = b.z; o[7] = b.w;
    }
    static __device__ __forceinline__ void store(float* p, const float* o) {
        *(float4*)p = make_float4(o[0], o[1], o[2], o[3]);
        *(float4*)(p + 4) = make_float4(o[4], o[5], o[6], o[7]);
    }
};

// bf16 element i (0..7) of 8 packed in a 16-byte register group, as float
__device__ __forceinline__ float bf16_lane(const u32x4& v, int i) {
    const uint32_t d = v[i >> 1];
    return __uint_as_float((i & 1) ? (d & 0xffff0000u) : (d << 16));
}

// Index of the sequence holding packed token t: the last s with cu[s] <= t (skips
// empty sequences). cu is monotone when valid; the search stays within [0, nseq-1].
__device__ __forceinline__ int seq_of(const int32_t* cu, int nseq, int64_t t) {
    int lo = 0, hi = nseq;  // invariant: answer in [lo, hi)
    while (hi - lo > 1) {
        int mid = (lo + hi) >> 1;
        if (cu[mid] <= t) lo = mid; else hi = mid;
    }
    return lo;
}

template <typename T, int K>
__global__ __launch_bounds__(256) void conv_prefill_kernel(ConvArgs a) {
    const int groups = a.E / kCV;
    // consecutive token runs on one XCD: the K-1 rows before a run are the end of the
    // previous run, fetched once into that XCD's L2
    const int64_t gid = (int64_t)xcd_contiguous((int)blockIdx.x, (int)gridDim.x) * blockDim.x + threadIdx.x;
    const int cg = (int)(gid % groups);
    const int64_t t0 = (gid / groups) * kTT;
    if (t0 >= a.T) return;
    const int c0 = cg * kCV;
    const T* xz = (const T*)a.xz;
    float w[kCV][K], bias[kCV];
#pragma unroll
    for (int i = 0; i < kCV; ++i) {
        bias[i] = to_f32(((const T*)a.b)[c0 + i]);
#pragma unroll
        for (int j = 0; j < K; ++j) w[i][j] = to_f32(((const T*)a.w)[(c0 + i) * K + j]);
    }
    int s = seq_of(a.cu, a.nseq, t0);
    int64_t s_begin = a.cu[s], s_end = a.cu[s + 1];
    const int64_t t1 = min(t0 + (int64_t)kTT, a.T);
    if constexpr (sizeof(T) == 2) {
        // a whole run inside one sequence whose K-1 earlier rows are inside it too (all but
        // the runs at sequence starts and ends): every input row of the run is requested
        // at once and kept as raw bf16, instead of one dependent load per token
        if (t1 - t0 == kTT && s_begin >= 0 && t0 - (K - 1) >= s_begin && t1 <= s_end) {
            u32x4 raw[kTT + K - 1];
#pragma unroll
            for (int r = 0; r < kTT + K - 1; ++r) raw[r] = *(const u32x4*)(xz + (t0 - (K - 1) + r) * a.ld_xz + c0);
#pragma unroll
            for (int t = 0; t < kTT; ++t) {
                float out[kCV];
#pragma unroll
                for (int i = 0; i < kCV; ++i) {
                    float acc = bias[i];
#pragma unroll
                    for (int j = 0; j < K; ++j) acc += w[i][j] * bf16_lane(raw[t + j], i);
                    out[i] = silu_f(acc);
                }
                Vec8<T>::store((T*)a.u + (t0 + t) * a.E + c0, out);
            }
            return;
        }
    }
    float win[K > 1 ? K - 1 : 1][kCV];  // previous K-1 inputs, oldest first
    bool fresh = true;
    for (int64_t t = t0; t < t1; ++t) {
        while (t >= s_end && s + 1 < a.nseq) {
            ++s; s_begin = a.cu[s]; s_end = a.cu[s + 1]; fresh = true;
        }
        if (t < s_begin || t >= s_end || s_begin < 0) {  // inconsistent cu_seqlens: leave u untouched
            atomicOr(a.status, SSM_STATUS_BAD_SEQLENS);
            fresh = true;
            continue;
        }
        if (fresh && K > 1) {
            // history positions t-(K-1) .. t-1 of the current sequence
            const int slot = a.slot[s];
            const bool init = a.has_init[s] != 0;
            const bool slot_ok = slot >= 0 && slot < a.S;
            if (init && !slot_ok) atomicOr(a.status, SSM_STATUS_BAD_SLOT);
#pragma unroll
            for (int j = 0; j < K - 1; ++j) {
                const int64_t p = t - (K - 1) + j;
                if (p >= s_begin) {
                    Vec8<T>::load(xz + p * a.ld_xz + c0, win[j]);
                } else if (init && slot_ok) {
                    const int hi = (int)(p - s_begin) + K - 1;  // index in the cached history
                    const T* h = (const T*)a.conv_pool + ((int64_t)slot * a.E + c0) * (K - 1) + hi;
#pragma unroll
                    for (int i = 0; i < kCV; ++i) win[j][i] = to_f32(h[i * (K - 1)]);
                } else {
#pragma unroll
                    for (int i = 0; i < kCV; ++i) win[j][i] = 0.0f;
                }
            }
        }
        fresh = false;
        float cur[kCV], out[kCV];
        Vec8<T>::load(xz + t * a.ld_xz + c0, cur);
#pragma unroll
        for (int i = 0; i < kCV; ++i) {
            float acc = bias[i];
#pragma unroll
            for (int j = 0; j < K - 1; ++j) acc += w[i][j] * win[j][i];
            acc += w[i][K - 1] * cur[i];
            out[i] = silu_f(acc);
        }
        Vec8<T>::store((T*)a.u + t * a.E + c0, out);
#pragma unroll
        for (int j = 0; j + 1 < K - 1; ++j)
#pragma unroll
            for (int i = 0; i < kCV; ++i) win[j][i] = win[j + 1][i];
        if (K > 1) {
#pragma unroll
            for (int i = 0; i < kCV; ++i) win[K > 1 ? K - 2 : 0][i] = cur[i];
        }
    }
}

// New history of each sequence = last K-1 entries of (old history | its inputs). Runs
// after the convolution has read the old histories; each thread reads all it needs
// before writing, so short pieces (fewer than K-1 tokens) keep the right old entries.
template <typename T, int K>
__global__ __launch_bounds__(256) void conv_state_update_kernel(ConvArgs a) {
    const int groups = a.E / kCV;
    const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (gid >= (int64_t)a.nseq * groups) return;
    const int s = (int)(gid / groups);
    const int c0 = (int)(gid % groups) * kCV;
    const int slot = a.slot[s];
    if (slot < 0 || slot >= a.S) {
        atomicOr(a.status, SSM_STATUS_BAD_SLOT);
        return;
    }
    const int64_t b = a.cu[s], e = a.cu[s + 1];
    if (b < 0 || e < b || e > a.T) {
        atomicOr(a.status, SSM_STATUS_BAD_SEQLENS);
        return;
    }
    const bool init = a.has_init[s] != 0;
    const int64_t L = e - b;
    T* hist = (T*)a.conv_pool + ((int64_t)slot * a.E + c0) * (K - 1);
    float nh[K > 1 ? K - 1 : 1][kCV];
#pragma unroll
    for (int i = 0; i < K - 1; ++i) {
        const int64_t p = e - (K - 1) + i;
        if (p >= b) {
            Vec8<T>::load((const T*)a.xz + p * a.ld_xz + c0, nh[i]);
        } else if (init) {
            const int oi = (int)(i + L);  // < K-1 here
#pragma unroll
            for (int c = 0; c < kCV; ++c) nh[i][c] = to_f32(hist[c * (K - 1) + oi]);
        } else {
#pragma unroll
            for (int c = 0; c < kCV; ++c) nh[i][c] = 0.0f;
        }
    }
#pragma unroll
    for (int i = 0; i < K - 1; ++i)
#pragma unroll
        for (int c = 0; c < kCV; ++c) hist[c * (K - 1) + i] = from_f32<T>(nh[i][c]);
}

template <typename T, int K>
__global__ __launch_bounds__(256) void conv_decode_kernel(ConvArgs a) {
    const int groups = a.E / kCV;
    const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (gid >= (int64_t)a.nseq * groups) return;
    const int bidx = (int)(gid / groups);
    const int c0 = (int)(gid % groups) * kCV;
    const int slot = a.slot[bidx];
    const bool slot_ok = slot >= 0 && slot < a.S;
    float cur[kCV], out[kCV];
    Vec8<T>::load((const T*)a.xz + (int64_t)bidx * a.ld_xz + c0, cur);
    // a bad slot still addresses slot 0 for the (discarded) history read
    T* hist = (T*)a.conv_pool + ((int64_t)(slot_ok ? slot : 0) * a.E + c0) * (K - 1);
    conv_window_step8<T, K>(cur, hist, slot_ok, (const T*)a.w + (int64_t)c0 * K, (const T*)a.b + c0, out);
    if (!slot_ok) atomicOr(a.status, SSM_STATUS_BAD_SLOT);
    Vec8<T>::store((T*)a.u + (int64_t)bidx * a.E + c0, out);
}

// Launch KERN<T, K> for the runtime width K (1..4) with one thread per work item.
#define SSM_CONV_LAUNCH(KERN, T, a, threads, s)                                              \
    do {                                                                                      \
        if ((threads) <= 0) return hipSuccess;                                                \
        const dim3 grid_((unsigned)(((threads) + 255) / 256)), block_(256);                  \
        switch ((a).K) {                                                                      \
            case 1: SSM_LAUNCH((KERN<T, 1>), grid_, block_, 0, s, a); break;         \
            case 2: SSM_LAUNCH((KERN<T, 2>), grid_, block_, 0, s, a); break;         \
            case 3: SSM_LAUNCH((KERN<T, 3>), grid_, block_, 0, s, a); break;         \
            default: SSM_LAUNCH((KERN<T, 4>), grid_, block_, 0, s, a); break;        \
        }                                                                                     \
        return hipGetLastError();                                                             \
    } while (0)

}  // namespace

hipError_t launch_conv_prefill(const ConvArgs& a, bool bf, hipStream_t s) {
    const int64_t threads = ((a.T + kTT - 1) / kTT) * (a.E / kCV);
    if (bf) SSM_CONV_LAUNCH(conv_prefill_kernel, bf16, a, threads, s);
    SSM_CONV_LAUNCH(conv_prefill_kernel, float, a, threads, s);
}
hipError_t launch_conv_state_update(const ConvArgs& a, bool bf, hipStream_t s) {
    if (a.K == 1) return hipSuccess;  // no history to keep
    const int64_t threads = (int64_t)a.nseq * (a.E / kCV);
    if (bf) SSM_CONV_LAUNCH(conv_state_update_kernel, bf16, a, threads, s);
    SSM_CONV_LAUNCH(conv_state_update_kernel, float, a, threads, s);
}
hipError_t launch_conv_decode(const ConvArgs& a, bool bf, hipStream_t s) {
    const int64_t threads = (int64_t)a.nseq * (a.E / kCV);
    if (bf) SSM_CONV_LAUNCH(conv_decode_kernel, bf16, a, threads, s);
    SSM_CONV_LAUNCH(conv_decode_kernel, float, a, threads, s);
}

}  // namespace ssm
