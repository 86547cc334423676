// Internal declarations shared by the gfx950 kernels and the C-ABI layer.
#pragma once
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "ssm_shard.h"

namespace ssm {

using bf16 = __bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

constexpr int kN = 16;          // states per channel the kernels are built for
constexpr int kMaxConv = 4;     // largest convolution width
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// Activation element <-> float. bf16 stores round to nearest even (hardware cvt on gfx950).
__device__ __forceinline__ float to_f32(float v) { return v; }
__device__ __forceinline__ float to_f32(bf16 v) { return (float)v; }
template <typename T> __device__ __forceinline__ T from_f32(float v);
template <> __device__ __forceinline__ float from_f32<float>(float v) { return v; }
template <> __device__ __forceinline__ bf16 from_f32<bf16>(float v) { return (bf16)v; }

// Raw buffer resource over [base, base + bytes): a load whose byte offset is at or beyond
// `bytes` returns zero and touches no memory, so bounds become offsets, not branches.
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
constexpr uint32_t kOffOutOfRange = 0x80000000u;  // an offset past any resource this library builds
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_rsrc(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}
__device__ __forceinline__ u32x4 buffer_load16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, 0);
}

// Global -> LDS on the DMA path: buffer_load_dwordx4 ... lds writes each lane's 16 bytes
// at lane slot (lane * 16) of a 1 KB LDS block at lds_addr (M0), with no staging
// registers. The source is the buffer resource r at byte offset voff (per lane) + soff
// (uniform), so a lane's offset stays fixed while soff walks along K; 32-bit offsets
// and a descriptor also keep the address unit's work below that of 64-bit flat
// addresses (the same tiles ran 3-8% faster than with global_load_lds_dwordx4).
// Issued from inline assembly so the compiler does not wait for it before unrelated LDS
// reads; completion is awaited with wait_vm (the wave's vector-memory counter).
typedef __attribute__((address_space(3))) void* lds_ptr_t;

#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void dma16(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff, uint32_t lds_addr) {
    asm volatile("s_mov_b32 m0, %3\n\tbuffer_load_dwordx4 %0, %1, %2 offen lds" ::"v"(voff), "s"(r), "s"(soff), "s"(lds_addr)
                 : "memory", "m0");
}
#pragma clang diagnostic pop

// wait until at most n of this wave's vector-memory loads are outstanding (n < 64).
// GFX9 s_waitcnt immediate: vmcnt in bits [3:0] and [15:14]; expcnt [6:4] and
// lgkmcnt [11:8] at their maxima (no wait on them).
template <int n> __device__ __forceinline__ void wait_vm() {
    static_assert(n >= 0 && n < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((n & 0xF) | ((n >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}
// wait until this wave's LDS reads (and other lgkm operations) are complete
__device__ __forceinline__ void wait_lgkm0() { __builtin_amdgcn_s_waitcnt(0xC07F); }

// exp2 / log2 on the transcendental unit (v_exp_f32 / v_log_f32).
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float fast_log2(float x) { return __builtin_amdgcn_logf(x); }
__device__ __forceinline__ float fast_rcp(float x) { return __builtin_amdgcn_rcpf(x); }

// softplus(v) = log(1 + e^v) = max(v, 0) + log1p(w) with w = e^-|v| in (0, 1]. With
// p = 1 + w rounded, p - 1 is exact and d = w - (p - 1) is the rounding error of p, so
// log1p(w) = log(p) + d / p to first order; p lies in (1, 2] and |d| is at most half an ulp
// of 1, so d / p may take 2 - p for 1 / p (an error of d (p - 1)^2 / p: about w^2 d for
// small w, at most d / 2 at w = 1, where log1p is 0.69). Two transcendentals (exp, log) and
// full relative accuracy for small w, as the usual log(p) * w / (p - 1) form of log1p gives
// with a third (the reciprocal).
__device__ __forceinline__ float softplus_f(float v) {
    const float w = fast_exp2(-fabsf(v) * kLog2e);
    const float p = 1.0f + w;
    const float d = w - (p - 1.0f);
    return fmaxf(v, 0.0f) + __builtin_fmaf(d, 2.0f - p, fast_log2(p) * kLn2);
}
// SiLU(v) = v / (1 + e^-v)
// min(rem, cap) for a row count, in integer arithmetic (the 64-bit min of the device headers
// is evaluated in double precision, which leaves the result in vector registers)
__device__ __forceinline__ int rows_upto(int64_t rem, int cap) { return rem < cap ? (int)rem : cap; }
__device__ __forceinline__ float silu_f(float v) { return v * fast_rcp(1.0f + fast_exp2(-v * kLog2e)); }

// Workgroups are dispatched round robin over the 8 XCDs (workgroup b on XCD b % 8). This
// maps b to a logical index so that each XCD gets one contiguous range of logical indices:
// neighbouring pieces of work that share input rows then share that XCD's L2. A bijection
// on [0, n) for any n.
__device__ __forceinline__ int xcd_contiguous(int b, int n) {
    const int per = n / 8, rem = n % 8, x = b % 8, i = b / 8;
    return x * per + (x < rem ? x : rem) + i;
}

// n elements at a 16-byte aligned address, as whole 16-byte loads and stores
template <typename T, int n> __device__ __forceinline__ void load16(const T* p, T (&o)[n]) {
    static_assert((n * sizeof(T)) % 16 == 0, "whole 16-byte pieces");
    u32x4 r[n * sizeof(T) / 16];
#pragma unroll
    for (int i = 0; i < (int)(n * sizeof(T) / 16); ++i) r[i] = ((const u32x4*)p)[i];
    __builtin_memcpy(o, r, sizeof o);
}
template <typename T, int n> __device__ __forceinline__ void store16(T* p, const T (&o)[n]) {
    static_assert((n * sizeof(T)) % 16 == 0, "whole 16-byte pieces");
    u32x4 r[n * sizeof(T) / 16];
    __builtin_memcpy(r, o, sizeof o);
#pragma unroll
    for (int i = 0; i < (int)(n * sizeof(T) / 16); ++i) ((u32x4*)p)[i] = r[i];
}

// One decode step of the cached convolution window (Section IV-A: the conv half of the
// cache) for 8 consecutive channels c0..c0+7 of one sequence: out = SiLU(b + sum_j w[j] *
// window), with cur (the new input, already in the activation dtype) as the newest tap,
// then the history [8][K-1] (oldest first) shifted by one with cur appended. The history
// (8 (K-1) elements), the weights [8][K] and the bias are contiguous 16-byte multiples at
// 16-byte aligned addresses (c0 % 8 == 0), so each is read and written in whole 16-byte
// pieces. load() fetches them; step() computes and writes the new history (ok false: the
// slot was bad, nothing is written and out is zero).
template <typename T, int K> struct ConvWindow8 {
    T wv[8 * K], bv[8], hv[K > 1 ? 8 * (K - 1) : 8];
    __device__ __forceinline__ void load(const T* hist, const T* w, const T* b) {
        load16(w, wv);
        load16(b, bv);
        if constexpr (K > 1) load16(hist, hv);
    }
    __device__ __forceinline__ void step(const float (&cur)[8], T* hist, bool ok, float (&out)[8]) const {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            float acc = to_f32(bv[i]);
#pragma unroll
            for (int j = 0; j < K - 1; ++j) acc += to_f32(wv[i * K + j]) * to_f32(hv[i * (K - 1) + j]);
            acc += to_f32(wv[i * K + K - 1]) * cur[i];
            out[i] = ok ? silu_f(acc) : 0.0f;
        }
        if constexpr (K > 1) {
            T nh[8 * (K - 1)];
#pragma unroll
            for (int i = 0; i < 8; ++i) {
#pragma unroll
                for (int j = 0; j + 1 < K - 1; ++j) nh[i * (K - 1) + j] = hv[i * (K - 1) + j + 1];
                nh[i * (K - 1) + K - 2] = from_f32<T>(cur[i]);
            }
            if (ok) store16(hist, nh);
        }
    }
};
template <typename T, int K>
__device__ __forceinline__ void conv_window_step8(const float (&cur)[8], T* hist, bool hist_ok, const T* w,
                                                  const T* b, float (&out)[8]) {
    ConvWindow8<T, K> cw;
    cw.load(hist, w, b);
    cw.step(cur, hist, hist_ok, out);
}

// Workspace header: status word at offset 0; regions start 256-byte aligned.
constexpr size_t kWsHeader = 256;
__host__ __device__ inline size_t align256(size_t b) { return (b + 255) & ~size_t(255); }

// ---------------------------------------------------------------- launchers
// GEMM: C[M][N] = A[M][K] * B[N][K]^T. Returns hipError_t of the launch. The role picks
// the kernel instance (each projection has its own symbol in profiles).
enum GemmRole { kGemmGeneric = 0, kGemmInProj = 1, kGemmXProj = 2, kGemmDtProj = 3, kGemmOutProj = 4 };
// o [M][K] bf16 (dense) = a [M][K] fp32 (row stride lda) rounded to nearest even; K % 8 == 0
hipError_t launch_round_bf16_rows(const float* a, int64_t lda, void* o, int64_t M, int K, hipStream_t s);
// scratch: fp32 partials of a split-K run (outputs with fewer tiles than CUs and a long
// K); gemm_splitk_bytes gives the size a shape would use (0: it is not split), and with
// less scratch the GEMM runs unsplit.
hipError_t launch_gemm_nt(int64_t M, int64_t N, int64_t K, const void* A, int64_t lda, int a_dt,
                          const void* B, int64_t ldb, int b_dt, void* C, int64_t ldc, int c_dt,
                          hipStream_t s, GemmRole role, float* scratch = nullptr, size_t scratch_bytes = 0);
size_t gemm_splitk_bytes(int64_t M, int64_t N, int64_t K, int a_dt, int b_dt, GemmRole role);
// Few-row (decode) GEMM C = A * B^T with a fused epilogue; bf16 weights.
enum SkinnyEpi { kSkinnyStoreBf16 = 0, kSkinnyStoreF32 = 1, kSkinnyConv = 2, kSkinnyState = 3 };
struct SkinnyArgs {
    const void* A; int64_t lda; bool a_f32;       // A [M][K], bf16 or fp32 (rounded to bf16 on load)
    const bf16* B; int64_t ldb;                   // B [N][K] bf16
    void* C; int64_t ldc;                         // plain stores
    int M, N, K;
    const int32_t* slot; int S; int32_t* status;  // per-row cache slot (fused epilogues)
    int E;                                        // channels of the shard
    // kSkinnyConv (in_proj): columns [conv_lo, conv_lo + conv_n) go through the cached conv
    // window (weights [conv_n][Kc], history pool [S][conv_n][Kc - 1]) into u [M][conv_n];
    // the other columns are stored to C in bf16
    const void* conv_w; const void* conv_b; void* conv_pool; int Kc; int conv_lo, conv_n; void* u;
    // kSkinnyState (dt_proj): B and C in xdbl, per-channel parameters, state pool, g out (u, z in)
    void* z; int64_t ld_z;
    const float* xdbl; int64_t ld_xdbl; int R; const float* b_dt; const float* A_log; const float* D;
    float* pool; void* g;
    // gated RMSNorm applied to A as it is loaded (Mamba-2 out_proj): column c of row m is
    // multiplied by 1 / sqrt(sumsq[m][k] / gsize + eps) and norm_w[c], k = (c0 + c) / gsize
    const float* nrm_sumsq; const float* nrm_w; int nrm_G, nrm_gsize, nrm_c0; float nrm_eps;
};
hipError_t launch_gemm_skinny(const SkinnyArgs& p, SkinnyEpi epi, hipStream_t s);
// the streamed kernel with the norm prologue above (plain bf16 stores); hipErrorNotSupported
// when the shape does not suit it (the caller then runs the norm and the product apart)
hipError_t launch_gemv_norm(const SkinnyArgs& p, hipStream_t s);
// Few-row product with float32 operands, C[M][N] = A[M][K] * B[N][K]^T in float32 (the
// decode projections of a float32 layer); role (GemmRole) only names the kernel instance.
// hipErrorNotSupported when the shape does not suit it (M > 64, K % 32, unaligned rows).
hipError_t launch_gemv_f32_stream(int role, int64_t M, int64_t N, int64_t K, const float* A, int64_t lda,
                                  const float* B, int64_t ldb, float* C, int64_t ldc, hipStream_t s);
// The decode in_proj of a float32 layer with the conv window in its epilogue: columns below
// conv_n of C = A B^T are channel n of the conv path, which takes its K - 1 cached inputs
// from conv_pool[slot[m]][n] (float32 [S][conv_n][K - 1]), writes u[m][n] = SiLU(window) and
// shifts the window; the other columns are stored to C. 2 <= K <= 4. gemv_f32_conv_fits says
// whether a shape suits it (else the caller runs the product and the conv kernel apart;
// launching it anyway returns hipErrorNotSupported).
struct F32ConvEpi {
    const int32_t* slot; int S; float* conv_pool; const float* w; const float* b; float* u; int conv_n; int K;
    int32_t* status;
};
bool gemv_f32_conv_fits(int64_t M, int64_t N, int64_t K, const float* A, int64_t lda, const float* B, int64_t ldb,
                        const F32ConvEpi& cv);
hipError_t launch_gemv_f32_conv(int64_t M, int64_t N, int64_t K, const float* A, int64_t lda, const float* B,
                                int64_t ldb, float* C, int64_t ldc, const F32ConvEpi& cv, hipStream_t s);

struct ConvArgs {
    const void* xz; int64_t ld_xz;     // SSM half in columns 0..E-1
    const void* w; const void* b;      // [E][K], [E]
    void* u;                           // [T][E]
    void* conv_pool;                   // [S][E][K-1]
    const int32_t* cu; const int32_t* slot; const int32_t* has_init;
    int32_t* status;
    int64_t T; int E, K, nseq, S;
};
hipError_t launch_conv_prefill(const ConvArgs& a, bool bf16_act, hipStream_t s);
hipError_t launch_conv_state_update(const ConvArgs& a, bool bf16_act, hipStream_t s);
hipError_t launch_conv_decode(const ConvArgs& a, bool bf16_act, hipStream_t s);

struct ScanArgs {
    const void* u; const void* dt; const void* z; int64_t ld_z;   // z: stride 2E
    const float* xdbl; int64_t ld_xdbl; int R;                     // B at R, C at R+N
    const float* b_dt; const float* A_log; const float* D;
    void* g;                                                       // [T][E]
    float* pool;                                                   // [S][E][N]
    const int32_t* cu; const int32_t* slot; const int32_t* has_init;
    int32_t* status;
    // decode with dt_proj fused into the state step: dt_proj weight [E][R] (act dtype);
    // delta is x_dbl's first R columns
    const void* w_dt;
    // scan scratch (prefill only)
    float* h_local; float* sum_delta; float* h_in; float* h0_seq;
    float* delta;                                                  // [T][E]: Delta of every token
    int64_t T; int E, nseq, S, win;                                // win: tokens per window
};
int scan_window_len(int64_t T, int E);
size_t scan_scratch_bytes(int64_t max_T, int E, int max_seqs);
hipError_t launch_scan_prefill(const ScanArgs& a, bool bf16_act, hipStream_t s);
hipError_t launch_decode_ssm(const ScanArgs& a, bool bf16_act, hipStream_t s);
// the same state step with dt = delta . W_dt^T computed in place of reading it (dt_rank a
// multiple of 8); hipErrorNotSupported otherwise
hipError_t launch_decode_dt_ssm(const ScanArgs& a, bool bf16_act, hipStream_t s);

// Names the launches made while it is alive; when timing is on (and the stream is not
// being captured into a graph), each of those launches is timed by the kernel's own
// dispatch timestamps (see launch_timed_events).
class KernelTimer {
  public:
    KernelTimer(const char* name, hipStream_t s);
    ~KernelTimer();
    KernelTimer(const KernelTimer&) = delete;
    KernelTimer& operator=(const KernelTimer&) = delete;

  private:
    const char* prev_;
};

// For a launch under an active KernelTimer: hands out a start/stop event pair that
// hipExtLaunchKernel binds to the dispatch itself (begin and end of the kernel, not of
// the queue position), and records it under the timer's name. False when not timing.
bool launch_timed_events(hipEvent_t* start, hipEvent_t* stop);

// Every kernel of the library is launched through this macro.
#define SSM_LAUNCH(K, grid, block, shm, s, ...)                                             \
    do {                                                                                    \
        hipEvent_t e0_, e1_;                                                                \
        if (::ssm::launch_timed_events(&e0_, &e1_))                                         \
            hipExtLaunchKernelGGL(K, grid, block, shm, s, e0_, e1_, 0, __VA_ARGS__);        \
        else                                                                                \
            hipLaunchKernelGGL(K, grid, block, shm, s, __VA_ARGS__);                        \
    } while (0)

// Mamba-2 (SSD) state update of one shard (ssd.hip); headdim 64, d_state 128, bf16.
struct SsdPublic {
    const void* zx; int64_t ld_zx;     // in_proj output [T][ld_zx]: z at col 0, dt at dt_col
    const void* u; int64_t ld_u;       // conv output [T][ld_u]: x at col 0, B at b_col, C at c_col
    int dt_col, b_col, c_col;
    int H;                             // heads of the shard
    int h_global0, hpg, g_off;         // first global head, heads per B/C group, local group offset
    const float* dt_bias; const float* A_log; const float* D;
    void* g; float* hs;                // [T][H*64] gated output; [T][H] sums of g^2 per head
    float* pool;                       // [S][H][64][128]
    const int32_t* cu; const int32_t* slot; const int32_t* has_init;
    int32_t* status;
    int nseq, S, win;
    int64_t T;
    void* plan; int32_t* plan_count; int max_windows;
    float* states; float* lsum;        // [max_windows][H][64][128], [max_windows][H]
};
int ssd_window_len(int64_t T, int H);
int ssd_max_windows(int64_t T, int nseq, int win);
size_t ssd_state_bytes(int max_windows, int H);
hipError_t launch_ssd_prefill(const SsdPublic& p, hipStream_t s);
hipError_t launch_ssd_decode(const SsdPublic& p, int batch, hipStream_t s);
hipError_t launch_ssd_group_sumsq(const float* hs, int H, int h_global0, int hpg, int G, float* out, int64_t T,
                                  hipStream_t s);
hipError_t launch_ssd_norm(const void* g, const float* sumsq, const float* norm_w, void* out, int64_t T, int E, int G,
                           int gsize, int c_global0, float eps, hipStream_t s);

// Quantized exchange payloads (codec.hip). codec: SSM_CODEC_*; cols % 8 == 0.
size_t codec_scale_bytes(int64_t rows);
size_t codec_payload_bytes(int codec, int64_t rows, int64_t cols);
hipError_t launch_codec_encode(int codec, const void* src, bool src_bf16, int64_t ld, int64_t rows, int64_t cols,
                               void* payload, hipStream_t s);
hipError_t launch_codec_decode_acc(int codec, const void* payload, int64_t rows, int64_t cols, float* acc, int64_t ld,
                                   bool accumulate, hipStream_t s);

hipError_t launch_fill_zero(void* p, int64_t bytes, hipStream_t s);  // bytes: multiple of 4
hipError_t launch_reduce_add(float* dst, const float* src, int64_t n, hipStream_t s);
hipError_t launch_copy_rows(void* dst, int64_t ld_dst, const void* src, int64_t ld_src,
                            int64_t rows, int64_t row_bytes, hipStream_t s);

// ---------------------------------------------------------------- layer (layer.hip)
constexpr int kMaxNormParts = 8;
struct NormParts {
    const void* p[kMaxNormParts];   // partial outputs added to the residual, in this order
    int n;
};
int residual_rmsnorm_max_dim();
hipError_t launch_residual_rmsnorm(const void* base, bool base_bf16, const NormParts& parts, bool parts_bf16,
                                   float* resid, const float* w, float eps, void* out, bool out_bf16, int64_t T, int d,
                                   hipStream_t s);
hipError_t launch_bcdt_rms(float* x, int64_t T, int R, int N, int64_t ld, float eps, hipStream_t s);

}  // namespace ssm
