// Quantized exchange payloads (Section IV-D: the remaining AllReduces carry a lower
// precision than the computation, FP16 from FP32 in the paper, and are converted back
// afterwards). A rank encodes its partial sum [rows][cols] into a payload; the receiver
// decodes each payload and adds it into an fp32 sum. Codecs:
//   f16 / bf16   element-wise, round to nearest even (v_cvt_f16_f32, v_cvt_pk_bf16_f32)
//   fp8          OCP E4M3 of x * (448 / max|row|) (v_cvt_pk_fp8_f32), one fp32 scale per row
//   int8         round-half-even of x * (127 / max|row|), one fp32 scale per row
// Payload: [rows] fp32 scales padded to 256 bytes (scaled codecs only), then the
// [rows][cols] codes, dense. Scales and products are computed in fp32, so a payload is a
// deterministic function of its input.
#include "common.h"

namespace ssm {
namespace {

constexpr int kF16 = 0, kBF16 = 1, kFP8 = 2, kI8 = 3;

template <typename T> struct Vec8;
template <> struct Vec8<float> {
    __device__ static void load(const float* p, float (&v)[8]) {
        const float4 a = ((const float4*)p)[0], b = ((const float4*)p)[1];
        v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w; v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
    }
};
template <> struct Vec8<bf16> {
    __device__ static void load(const bf16* p, float (&v)[8]) {
        const bf16x8 a = *(const bf16x8*)p;
#pragma unroll
        for (int i = 0; i < 8; ++i) v[i] = (float)a[i];
    }
};

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));

// ---------------------------------------------------------------- element-wise codecs
template <typename T, int CODEC>
__global__ __launch_bounds__(256) void encode_elem_kernel(const T* __restrict__ src, int64_t ld, int64_t rows,
                                                          int64_t cols, uint16_t* __restrict__ out) {
    const int64_t g8 = cols / 8;
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= rows * g8) return;
    const int64_t r = i / g8, c = (i % g8) * 8;
    float v[8];
    Vec8<T>::load(src + r * ld + c, v);
    uint16_t* o = out + r * cols + c;
    if constexpr (CODEC == kF16) {
        f16x8 h;
#pragma unroll
        for (int k = 0; k < 8; ++k) h[k] = (_Float16)v[k];
        *(f16x8*)o = h;
    } else {
        bf16x8 h;
#pragma unroll
        for (int k = 0; k < 8; ++k) h[k] = (bf16)v[k];
        *(bf16x8*)o = h;
    }
}

// ---------------------------------------------------------------- row-scaled codecs
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, 64));
    return v;
}

// 8 scaled values -> 8 codes (one 64-bit word)
template <int CODEC>
__device__ __forceinline__ uint2 quantize8(const float (&v)[8], float inv) {
    constexpr float Q = CODEC == kFP8 ? 448.0f : 127.0f;
    float q[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) q[k] = fminf(fmaxf(v[k] * inv, -Q), Q);
    uint32_t w[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        if constexpr (CODEC == kFP8) {
            int p = __builtin_amdgcn_cvt_pk_fp8_f32(q[4 * h], q[4 * h + 1], 0, false);
            p = __builtin_amdgcn_cvt_pk_fp8_f32(q[4 * h + 2], q[4 * h + 3], p, true);
            w[h] = (uint32_t)p;
        } else {
            uint32_t x = 0;
#pragma unroll
            for (int k = 0; k < 4; ++k) x |= ((uint32_t)(int32_t)__builtin_rintf(q[4 * h + k]) & 0xFFu) << (8 * k);
            w[h] = x;
        }
    }
    return make_uint2(w[0], w[1]);
}

// One wave per row. Rows of up to NCH * 512 values stay in registers between the amax
// pass and the quantize pass (NCH = 0: any length, the row is read twice).
template <typename T, int CODEC, int NCH>
__global__ __launch_bounds__(256) void encode_scaled_kernel(const T* __restrict__ src, int64_t ld, int64_t rows,
                                                            int64_t cols, float* __restrict__ scales,
                                                            uint8_t* __restrict__ codes) {
    constexpr float Q = CODEC == kFP8 ? 448.0f : 127.0f;
    const int lane = threadIdx.x & 63;
    const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (r >= rows) return;
    const T* row = src + r * ld;
    uint8_t* crow = codes + r * cols;
    float amax = 0.0f;
    if constexpr (NCH > 0) {
        float v[NCH][8];
#pragma unroll
        for (int j = 0; j < NCH; ++j) {
            const int64_t c = (int64_t)(j * 64 + lane) * 8;
            if (c < cols) {
                Vec8<T>::load(row + c, v[j]);
#pragma unroll
                for (int k = 0; k < 8; ++k) amax = fmaxf(amax, fabsf(v[j][k]));
            }
        }
        amax = wave_max(amax);
        const float inv = amax > 0.0f ? Q / amax : 0.0f;
#pragma unroll
        for (int j = 0; j < NCH; ++j) {
            const int64_t c = (int64_t)(j * 64 + lane) * 8;
            if (c < cols) *(uint2*)(crow + c) = quantize8<CODEC>(v[j], inv);
        }
    } else {
        for (int64_t c = (int64_t)lane * 8; c < cols; c += 512) {
            float v[8];
            Vec8<T>::load(row + c, v);
#pragma unroll
            for (int k = 0; k < 8; ++k) amax = fmaxf(amax, fabsf(v[k]));
        }
        amax = wave_max(amax);
        const float inv = amax > 0.0f ? Q / amax : 0.0f;
        for (int64_t c = (int64_t)lane * 8; c < cols; c += 512) {
            float v[8];
            Vec8<T>::load(row + c, v);
            *(uint2*)(crow + c) = quantize8<CODEC>(v, inv);
        }
    }
    if (lane == 0) scales[r] = amax / Q;
}

// ---------------------------------------------------------------- decode + accumulate
template <int CODEC>
__device__ __forceinline__ void decode8(const void* codes, int64_t off, float s, float (&v)[8]) {
    if constexpr (CODEC == kF16) {
        const f16x8 h = *(const f16x8*)((const uint16_t*)codes + off);
#pragma unroll
        for (int k = 0; k < 8; ++k) v[k] = (float)h[k];
    } else if constexpr (CODEC == kBF16) {
        const bf16x8 h = *(const bf16x8*)((const uint16_t*)codes + off);
#pragma unroll
        for (int k = 0; k < 8; ++k) v[k] = (float)h[k];
    } else {
        const uint2 w = *(const uint2*)((const uint8_t*)codes + off);
        const uint32_t ww[2] = {w.x, w.y};
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            if constexpr (CODEC == kFP8) {
                v[4 * h + 0] = __builtin_amdgcn_cvt_f32_fp8((int)ww[h], 0) * s;
                v[4 * h + 1] = __builtin_amdgcn_cvt_f32_fp8((int)ww[h], 1) * s;
                v[4 * h + 2] = __builtin_amdgcn_cvt_f32_fp8((int)ww[h], 2) * s;
                v[4 * h + 3] = __builtin_amdgcn_cvt_f32_fp8((int)ww[h], 3) * s;
            } else {
#pragma unroll
                for (int k = 0; k < 4; ++k) v[4 * h + k] = (float)(int8_t)((ww[h] >> (8 * k)) & 0xFF) * s;
            }
        }
    }
}

template <int CODEC>
__global__ __launch_bounds__(256) void decode_acc_kernel(const float* __restrict__ scales, const void* __restrict__ codes,
                                                         int64_t rows, int64_t cols, float* __restrict__ acc,
                                                         int64_t ld, int accumulate) {
    const int64_t g8 = cols / 8;
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= rows * g8) return;
    const int64_t r = i / g8, c = (i % g8) * 8;
    const float s = (CODEC == kFP8 || CODEC == kI8) ? scales[r] : 1.0f;
    float v[8];
    decode8<CODEC>(codes, r * cols + c, s, v);
    float4* a = (float4*)(acc + r * ld + c);
    if (accumulate) {
        const float4 x = a[0], y = a[1];
        v[0] += x.x; v[1] += x.y; v[2] += x.z; v[3] += x.w; v[4] += y.x; v[5] += y.y; v[6] += y.z; v[7] += y.w;
    }
    a[0] = make_float4(v[0], v[1], v[2], v[3]);
    a[1] = make_float4(v[4], v[5], v[6], v[7]);
}

unsigned grid8(int64_t rows, int64_t cols) { return (unsigned)((rows * (cols / 8) + 255) / 256); }

template <typename T, int CODEC>
void launch_scaled(const T* src, int64_t ld, int64_t rows, int64_t cols, float* scales, uint8_t* codes,
                   hipStream_t s) {
    const dim3 grid((unsigned)((rows + 3) / 4)), block(256);
    if (cols <= 512) SSM_LAUNCH((encode_scaled_kernel<T, CODEC, 1>), grid, block, 0, s, src, ld, rows, cols, scales, codes);
    else if (cols <= 1024) SSM_LAUNCH((encode_scaled_kernel<T, CODEC, 2>), grid, block, 0, s, src, ld, rows, cols, scales, codes);
    else if (cols <= 2048) SSM_LAUNCH((encode_scaled_kernel<T, CODEC, 4>), grid, block, 0, s, src, ld, rows, cols, scales, codes);
    else if (cols <= 4096) SSM_LAUNCH((encode_scaled_kernel<T, CODEC, 8>), grid, block, 0, s, src, ld, rows, cols, scales, codes);
    else SSM_LAUNCH((encode_scaled_kernel<T, CODEC, 0>), grid, block, 0, s, src, ld, rows, cols, scales, codes);
}

template <typename T>
hipError_t encode_t(int codec, const T* src, int64_t ld, int64_t rows, int64_t cols, void* payload, hipStream_t s) {
    const unsigned g = grid8(rows, cols);
    switch (codec) {
        case kF16: SSM_LAUNCH((encode_elem_kernel<T, kF16>), dim3(g), dim3(256), 0, s, src, ld, rows, cols, (uint16_t*)payload); break;
        case kBF16: SSM_LAUNCH((encode_elem_kernel<T, kBF16>), dim3(g), dim3(256), 0, s, src, ld, rows, cols, (uint16_t*)payload); break;
        case kFP8:
            launch_scaled<T, kFP8>(src, ld, rows, cols, (float*)payload, (uint8_t*)payload + codec_scale_bytes(rows), s);
            break;
        default:
            launch_scaled<T, kI8>(src, ld, rows, cols, (float*)payload, (uint8_t*)payload + codec_scale_bytes(rows), s);
            break;
    }
    return hipGetLastError();
}

}  // namespace

size_t codec_scale_bytes(int64_t rows) { return align256((size_t)rows * 4); }

size_t codec_payload_bytes(int codec, int64_t rows, int64_t cols) {
    const size_t n = (size_t)rows * (size_t)cols;
    return (codec == kFP8 || codec == kI8) ? codec_scale_bytes(rows) + n : 2 * n;
}

hipError_t launch_codec_encode(int codec, const void* src, bool src_bf16, int64_t ld, int64_t rows, int64_t cols,
                               void* payload, hipStream_t s) {
    if (rows <= 0 || cols <= 0) return hipSuccess;
    return src_bf16 ? encode_t<bf16>(codec, (const bf16*)src, ld, rows, cols, payload, s)
                    : encode_t<float>(codec, (const float*)src, ld, rows, cols, payload, s);
}

hipError_t launch_codec_decode_acc(int codec, const void* payload, int64_t rows, int64_t cols, float* acc, int64_t ld,
                                   bool accumulate, hipStream_t s) {
    if (rows <= 0 || cols <= 0) return hipSuccess;
    const unsigned g = grid8(rows, cols);
    const float* sc = (const float*)payload;
    const void* codes = (codec == kFP8 || codec == kI8) ? (const void*)((const char*)payload + codec_scale_bytes(rows))
                                                          : payload;
    const int a = accumulate ? 1 : 0;
    switch (codec) {
        case kF16: SSM_LAUNCH((decode_acc_kernel<kF16>), dim3(g), dim3(256), 0, s, sc, codes, rows, cols, acc, ld, a); break;
        case kBF16: SSM_LAUNCH((decode_acc_kernel<kBF16>), dim3(g), dim3(256), 0, s, sc, codes, rows, cols, acc, ld, a); break;
        case kFP8: SSM_LAUNCH((decode_acc_kernel<kFP8>), dim3(g), dim3(256), 0, s, sc, codes, rows, cols, acc, ld, a); break;
        default: SSM_LAUNCH((decode_acc_kernel<kI8>), dim3(g), dim3(256), 0, s, sc, codes, rows, cols, acc, ld, a); break;
    }
    return hipGetLastError();
}

}  // namespace ssm
