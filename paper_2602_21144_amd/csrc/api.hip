// C ABI of the mixer shard: argument checks (host only, before anything is enqueued),
// workspace layout and the order of kernels for prefill and decode.
//
// Prefill (Section II-B order; Section IV-B reductions):
//   stage 1: in_proj GEMM -> xz; conv1d+SiLU -> u (and the conv history); x_proj GEMM -> x_dbl
//   [first reduction over shards: the caller's]
//   stage 2: dt_proj GEMM -> dt; selective scan -> g (and the final states); out_proj GEMM -> y
// Decode: the same with one token per sequence and the single-step kernels.
#include <algorithm>
#include <atomic>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "common.h"

using namespace ssm;

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_err = buf;
    return code;
}

int hip_fail(hipError_t e, const char* what) {
    return fail(SSM_E_HIP, "%s: %s", what, hipGetErrorString(e));
}

#define SSM_TRY_HIP(expr, what)                          \
    do {                                                 \
        hipError_t e_ = (expr);                          \
        if (e_ != hipSuccess) return hip_fail(e_, what); \
    } while (0)

#define SSM_TRY(expr)            \
    do {                         \
        int r_ = (expr);         \
        if (r_ != SSM_OK) return r_; \
    } while (0)

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

size_t act_bytes(const ssm_shard_desc_t* d) { return d->act_dtype == SSM_BF16 ? 2 : 4; }

int check_desc(const ssm_shard_desc_t* d) {
    if (!d) return fail(SSM_E_INVAL, "desc is null");
    if (d->act_dtype != SSM_F32 && d->act_dtype != SSM_BF16) return fail(SSM_E_INVAL, "act_dtype %d", d->act_dtype);
    if (d->d_model <= 0 || d->d_model % 16) return fail(SSM_E_INVAL, "d_model %d must be a positive multiple of 16", d->d_model);
    if (d->d_inner_shard <= 0 || d->d_inner_shard % 64)
        return fail(SSM_E_INVAL, "d_inner_shard %d must be a positive multiple of 64", d->d_inner_shard);
    if (d->shard_count <= 0 || d->shard_index < 0 || d->shard_index >= d->shard_count)
        return fail(SSM_E_INVAL, "shard %d of %d", d->shard_index, d->shard_count);
    if ((int64_t)d->d_inner_shard * d->shard_count != d->d_inner_total)
        return fail(SSM_E_INVAL, "d_inner_shard %d * shard_count %d != d_inner_total %d", d->d_inner_shard,
                    d->shard_count, d->d_inner_total);
    if (d->d_state != kN) return fail(SSM_E_INVAL, "d_state %d: the kernels are built for %d", d->d_state, kN);
    if (d->dt_rank <= 0 || d->dt_rank % 16) return fail(SSM_E_INVAL, "dt_rank %d must be a positive multiple of 16", d->dt_rank);
    if (d->d_conv < 1 || d->d_conv > kMaxConv) return fail(SSM_E_INVAL, "d_conv %d not in [1, %d]", d->d_conv, kMaxConv);
    return SSM_OK;
}

int check_weights(const ssm_shard_weights_t* w) {
    if (!w) return fail(SSM_E_INVAL, "weights is null");
    const void* ps[] = {w->in_proj_w, w->conv_w, w->conv_b, w->x_proj_w, w->dt_proj_w,
                        w->out_proj_w, w->dt_proj_b, w->A_log, w->D};
    const char* names[] = {"in_proj_w", "conv_w", "conv_b", "x_proj_w", "dt_proj_w",
                           "out_proj_w", "dt_proj_b", "A_log", "D"};
    for (int i = 0; i < 9; ++i) {
        if (!ps[i]) return fail(SSM_E_INVAL, "weights.%s is null", names[i]);
        if (!aligned16(ps[i])) return fail(SSM_E_ALIGN, "weights.%s is not 16-byte aligned", names[i]);
    }
    return SSM_OK;
}

int check_ptr(const void* p, const char* name) {
    if (!p) return fail(SSM_E_INVAL, "%s is null", name);
    if (!aligned16(p)) return fail(SSM_E_ALIGN, "%s is not 16-byte aligned", name);
    return SSM_OK;
}

int check_meta(const ssm_seq_meta_t* m, int64_t T) {
    if (!m) return fail(SSM_E_INVAL, "meta is null");
    if (m->nseq < 0) return fail(SSM_E_INVAL, "nseq %d", m->nseq);
    if (m->nseq == 0 && T != 0) return fail(SSM_E_SEQLENS, "T = %lld tokens but no sequences", (long long)T);
    if (m->nseq > 0 && (!m->cu_seqlens || !m->cache_slot || !m->has_initial_state))
        return fail(SSM_E_INVAL, "meta arrays must be non-null");
    return SSM_OK;
}

// ------------------------------------------------------------------ workspaces
// fp32 partials of the projections that run split-K (few tokens)
struct Scratch {
    float* p = nullptr;
    size_t bytes = 0;
};

struct PrefillWs {
    int32_t* status;
    char *xz, *u, *dt, *g;
    char* delta16;  // [T][R] bf16: delta rounded for dt_proj (bf16 activations)
    float* xdbl;
    char* scan;
    Scratch splitk;  // fp32 partials of the projections that run split-K (few tokens)
    size_t total;
};

PrefillWs prefill_layout(const ssm_shard_desc_t* d, int64_t T, int nseq, void* base) {
    const size_t s = act_bytes(d);
    const int64_t E = d->d_inner_shard, W = d->dt_rank + 2 * d->d_state;
    PrefillWs L{};
    char* b = (char*)base;
    size_t off = kWsHeader;
    auto take = [&](size_t bytes) { char* p = b ? b + off : nullptr; off += align256(bytes); return p; };
    L.status = (int32_t*)b;
    L.xz = take((size_t)T * 2 * E * s);
    L.u = take((size_t)T * E * s);
    L.xdbl = (float*)take((size_t)T * W * 4);
    L.dt = take((size_t)T * E * s);
    L.g = take((size_t)T * E * s);
    L.delta16 = take(d->act_dtype == SSM_BF16 ? (size_t)T * d->dt_rank * 2 : 0);
    L.scan = take(scan_scratch_bytes(T, (int)E, nseq));
    const int adt = d->act_dtype;
    const int64_t dm = d->d_model, R = d->dt_rank;
    size_t sk = gemm_splitk_bytes(T, 2 * E, dm, adt, adt, kGemmInProj);
    sk = std::max(sk, gemm_splitk_bytes(T, W, E, adt, adt, kGemmXProj));
    sk = std::max(sk, gemm_splitk_bytes(T, E, R, adt, adt, kGemmDtProj));
    sk = std::max(sk, gemm_splitk_bytes(T, dm, E, adt, adt, kGemmOutProj));
    L.splitk.p = (float*)take(sk);
    L.splitk.bytes = sk;
    L.total = off;
    return L;
}

struct DecodeWs {
    int32_t* status;
    char *xz, *u, *dt, *g;
    float* xdbl;
    Scratch splitk;  // fp32 partials of the projections that run split-K (large batches)
    size_t total;
};

// Largest decode batch whose dt_proj takes the state step in its epilogue (each workgroup
// of that kernel reads every activation row, which suits a few rows); larger batches run
// the state-step kernel with four lanes per (sequence, channel) and dt_proj folded in.
// Measured on the 2.8B quarter shard: the epilogue form faster at 64 sequences, the
// state-step kernel at 128.
constexpr int kFusedDecodeMax = 64;
// Largest bf16 decode batch whose in_proj takes the conv step in its epilogue: the
// streamed projection kernels cover up to 512 rows (16-row tiles, then tiles of 32 or 64
// rows over 32 columns).
constexpr int kConvEpilogueMax = 512;

DecodeWs decode_layout(const ssm_shard_desc_t* d, int64_t B, void* base) {
    const size_t s = act_bytes(d);
    const int64_t E = d->d_inner_shard, W = d->dt_rank + 2 * d->d_state;
    DecodeWs L{};
    char* b = (char*)base;
    size_t off = kWsHeader;
    auto take = [&](size_t bytes) { char* p = b ? b + off : nullptr; off += align256(bytes); return p; };
    L.status = (int32_t*)b;
    L.xz = take((size_t)B * 2 * E * s);
    L.u = take((size_t)B * E * s);
    L.xdbl = (float*)take((size_t)B * W * 4);
    L.dt = take((size_t)B * E * s);
    L.g = take((size_t)B * E * s);
    const int adt = d->act_dtype;
    const int64_t dm = d->d_model;
    size_t sk = 0;
    if (B > kFusedDecodeMax) {
        sk = gemm_splitk_bytes(B, 2 * E, dm, adt, adt, kGemmInProj);
        sk = std::max(sk, gemm_splitk_bytes(B, W, E, adt, adt, kGemmXProj));
        sk = std::max(sk, gemm_splitk_bytes(B, dm, E, adt, adt, kGemmOutProj));
    }
    L.splitk.p = (float*)take(sk);
    L.splitk.bytes = sk;
    L.total = off;
    return L;
}

int check_ws(void* ws, size_t have, size_t need) {
    if (!ws) return fail(SSM_E_INVAL, "workspace is null");
    if (!aligned16(ws)) return fail(SSM_E_ALIGN, "workspace is not 16-byte aligned");
    if (have < need) return fail(SSM_E_WORKSPACE, "workspace %zu bytes < %zu needed", have, need);
    return SSM_OK;
}

int gemm(int64_t M, int64_t N, int64_t K, const void* A, int64_t lda, int adt, const void* B, int64_t ldb, int bdt,
         void* C, int64_t ldc, int cdt, hipStream_t s, const char* what, GemmRole role = kGemmGeneric,
         Scratch sk = Scratch{}) {
    KernelTimer kt(what, s);
    SSM_TRY_HIP(launch_gemm_nt(M, N, K, A, lda, adt, B, ldb, bdt, C, ldc, cdt, s, role, sk.p, sk.bytes), what);
    return SSM_OK;
}

// one timed launch of a non-GEMM kernel
#define SSM_TIMED(name, s, expr)                 \
    do {                                         \
        KernelTimer kt_(name, s);                \
        SSM_TRY_HIP((expr), name);               \
    } while (0)

ConvArgs conv_args(const ssm_shard_desc_t* d, const ssm_shard_weights_t* w, const void* xz, int64_t T,
                   const int32_t* cu, const int32_t* slot, const int32_t* hi, int nseq, void* conv_pool, int S,
                   void* u, int32_t* status) {
    ConvArgs a{};
    a.xz = xz; a.ld_xz = 2 * (int64_t)d->d_inner_shard;
    a.w = w->conv_w; a.b = w->conv_b; a.u = u; a.conv_pool = conv_pool;
    a.cu = cu; a.slot = slot; a.has_init = hi; a.status = status;
    a.T = T; a.E = d->d_inner_shard; a.K = d->d_conv; a.nseq = nseq; a.S = S;
    return a;
}

ScanArgs scan_args(const ssm_shard_desc_t* d, const ssm_shard_weights_t* w, const void* u, const void* dt,
                   const void* xz, const float* xdbl, int64_t T, const int32_t* cu, const int32_t* slot,
                   const int32_t* hi, int nseq, float* pool, int S, void* g, int32_t* status, void* scratch) {
    ScanArgs a{};
    const int64_t E = d->d_inner_shard;
    a.u = u; a.dt = dt;
    a.z = (const char*)xz + E * act_bytes(d); a.ld_z = 2 * E;
    a.xdbl = xdbl; a.ld_xdbl = d->dt_rank + 2 * d->d_state; a.R = d->dt_rank;
    a.b_dt = w->dt_proj_b; a.A_log = w->A_log; a.D = w->D;
    a.g = g; a.pool = pool; a.cu = cu; a.slot = slot; a.has_init = hi; a.status = status;
    a.h_local = (float*)scratch;
    a.T = T; a.E = (int)E; a.nseq = nseq; a.S = S;
    a.win = scan_window_len(T, (int)E);
    return a;
}

int common_checks(const ssm_shard_desc_t* d, const ssm_shard_weights_t* w, int64_t T, int32_t S) {
    SSM_TRY(check_desc(d));
    SSM_TRY(check_weights(w));
    if (T < 0 || T > INT32_MAX) return fail(SSM_E_INVAL, "token count %lld", (long long)T);
    if (S <= 0) return fail(SSM_E_INVAL, "num_slots %d", S);
    return SSM_OK;
}

// stage bodies (arguments already checked)
int prefill1(const ssm_shard_desc_t* d, const ssm_shard_weights_t* w, const void* x, int64_t T,
             const ssm_seq_meta_t* m, void* conv_pool, int32_t S, float* xdbl, const PrefillWs& L, hipStream_t s) {
    const int adt = d->act_dtype;
    const int64_t E = d->d_inner_shard, W = d->dt_rank + 2 * d->d_state, dm = d->d_model;
    SSM_TRY(gemm(T, 2 * E, dm, x, dm, adt, w->in_proj_w, dm, adt, L.xz, 2 * E, adt, s, "prefill.in_proj", kGemmInProj, L.splitk));
    ConvArgs ca = conv_args(d, w, L.xz, T, m->cu_seqlens, m->cache_slot, m->has_initial_state, m->nseq, conv_pool,
                            S, L.u, L.status);
    SSM_TIMED("prefill.conv1d", s, launch_conv_prefill(ca, adt == SSM_BF16, s));
    SSM_TIMED("prefill.conv_history", s, launch_conv_state_update(ca, adt == SSM_BF16, s));
    SSM_TRY(gemm(T, W, E, L.u, E, adt, w->x_proj_w, E, adt, xdbl, W, SSM_F32, s, "prefill.x_proj", kGemmXProj, L.splitk));
    return SSM_OK;
}

int prefill2(const ssm_shard_desc_t* d, const ssm_shard_weights_t* w, const float* xdbl, int64_t T,
             const ssm_seq_meta_t* m, float* ssm_pool, int32_t S, void* y, const PrefillWs& L, hipStream_t s) {
    const int adt = d->act_dtype;
    const int64_t E = d->d_inner_shard, W = d->dt_rank + 2 * d->d_state, dm = d->d_model, R = d->dt_rank;
    if (adt == SSM_BF16 && R % 32 == 0 && T > 64) {
        // delta is rounded to bf16 once, so dt_proj runs on the DMA-fed bf16 tiles
        SSM_TIMED("prefill.dt_round", s, launch_round_bf16_rows(xdbl, W, L.delta16, T, (int)R, s));
        SSM_TRY(gemm(T, E, R, L.delta16, R, adt, w->dt_proj_w, R, adt, L.dt, E, adt, s, "prefill.dt_proj", kGemmDtProj, L.splitk));
    } else {
        SSM_TRY(gemm(T, E, R, xdbl, W, SSM_F32, w->dt_proj_w, R, adt, L.dt, E, adt, s, "prefill.dt_proj", kGemmDtProj, L.splitk));
    }
    ScanArgs sa = scan_args(d, w, L.u, L.dt, L.xz, xdbl, T, m->cu_seqlens, m->cache_slot, m->has_initial_state,
                            m->nseq, ssm_pool, S, L.g, L.status, L.scan);
    SSM_TRY_HIP(launch_scan_prefill(sa, adt == SSM_BF16, s), "selective scan");
    SSM_TRY(gemm(T, dm, E, L.g, E, adt, w->out_proj_w, E, adt, y, dm, adt, s, "prefill.out_proj", kGemmOutProj, L.splitk));
    return SSM_OK;
}

SkinnyArgs skinny(const void* A, int64_t lda, bool a_f32, const void* B, int64_t ldb, void* C, int64_t ldc, int64_t M,
                  int64_t N, int64_t K) {
    SkinnyArgs p{};
    p.A = A; p.lda = lda; p.a_f32 = a_f32; p.B = (const bf16*)B; p.ldb = ldb; p.C = C; p.ldc = ldc;
    p.M = (int)M; p.N = (int)N; p.K = (int)K;
    return p;
}

#define SSM_SKINNY(name, s, p, epi) SSM_TIMED(name, s, launch_gemm_skinny(p, epi, s))

int decode1(const ssm_shard_desc_t* d, const ssm_shard_weights_t* w, const void* x, int32_t B, const int32_t* slot,
            void* conv_pool, int32_t S, float* xdbl, const DecodeWs& L, hipStream_t s) {
    const int adt = d->act_dtype;
    const int64_t E = d->d_inner_shard, W = d->dt_rank + 2 * d->d_state, dm = d->d_model;
    if (adt == SSM_BF16 && d->d_conv >= 2 && B <= kConvEpilogueMax) {
        // in_proj with the conv window shift + SiLU fused into its epilogue; x_proj
        SkinnyArgs p = skinny(x, dm, false, w->in_proj_w, dm, L.xz, 2 * E, B, 2 * E, dm);
        p.slot = slot; p.S = S; p.status = L.status; p.E = (int)E;
        p.conv_w = w->conv_w; p.conv_b = w->conv_b; p.conv_pool = conv_pool; p.Kc = d->d_conv;
        p.conv_lo = 0; p.conv_n = (int)E; p.u = L.u;
        SkinnyArgs q = skinny(L.u, E, false, w->x_proj_w, E, xdbl, W, B, W, E);
        SSM_SKINNY("decode.in_proj_conv", s, p, kSkinnyConv);
        SSM_SKINNY("decode.x_proj", s, q, kSkinnyStoreF32);
        return SSM_OK;
    }
    if (adt == SSM_F32 && d->d_conv >= 2) {
        // float32: in_proj with the conv window in the streamed kernel's epilogue (up to 64
        // sequences; otherwise the product and the conv kernel below)
        const F32ConvEpi cv{slot, S, (float*)conv_pool, (const float*)w->conv_w, (const float*)w->conv_b,
                            (float*)L.u, (int)E, d->d_conv, L.status};
        const float* xf = (const float*)x;
        const float* wf = (const float*)w->in_proj_w;
        if (gemv_f32_conv_fits(B, 2 * E, dm, xf, dm, wf, dm, cv)) {
            SSM_TIMED("decode.in_proj_conv", s, launch_gemv_f32_conv(B, 2 * E, dm, xf, dm, wf, dm, (float*)L.xz, 2 * E, cv, s));
            SSM_TRY(gemm(B, W, E, L.u, E, adt, w->x_proj_w, E, adt, xdbl, W, SSM_F32, s, "decode.x_proj", kGemmXProj,
                         L.splitk));
            return SSM_OK;
        }
    }
    ConvArgs ca = conv_args(d, w, L.xz, B, nullptr, slot, nullptr, B, conv_pool, S, L.u, L.status);
    SSM_TRY(gemm(B, 2 * E, dm, x, dm, adt, w->in_proj_w, dm, adt, L.xz, 2 * E, adt, s, "decode.in_proj",
                 kGemmInProj, L.splitk));
    SSM_TIMED("decode.conv", s, launch_conv_decode(ca, adt == SSM_BF16, s));
    SSM_TRY(gemm(B, W, E, L.u, E, adt, w->x_proj_w, E, adt, xdbl, W, SSM_F32, s, "decode.x_proj", kGemmXProj,
                 L.splitk));
    return SSM_OK;
}

int decode2(const ssm_shard_desc_t* d, const ssm_shard_weights_t* w, const float* xdbl, int32_t B,
            const int32_t* slot, float* ssm_pool, int32_t S, void* y, const DecodeWs& L, hipStream_t s) {
    const int adt = d->act_dtype;
    const int64_t E = d->d_inner_shard, W = d->dt_rank + 2 * d->d_state, dm = d->d_model, R = d->dt_rank;
    if (adt == SSM_BF16 && B <= kFusedDecodeMax) {
        // dt_proj with the whole recurrence step fused into its epilogue; out_proj
        SkinnyArgs p = skinny(xdbl, W, true, w->dt_proj_w, R, nullptr, 0, B, E, R);
        p.slot = slot; p.S = S; p.status = L.status; p.E = (int)E;
        p.u = L.u; p.z = L.xz + E * act_bytes(d); p.ld_z = 2 * E;
        p.xdbl = xdbl; p.ld_xdbl = W; p.R = (int)R; p.b_dt = w->dt_proj_b; p.A_log = w->A_log; p.D = w->D;
        p.pool = ssm_pool; p.g = L.g;
        SkinnyArgs q = skinny(L.g, E, false, w->out_proj_w, E, y, dm, B, dm, E);
        SSM_SKINNY("decode.dt_proj_state", s, p, kSkinnyState);
        SSM_SKINNY("decode.out_proj", s, q, kSkinnyStoreBf16);
        return SSM_OK;
    }
    ScanArgs sa = scan_args(d, w, L.u, L.dt, L.xz, xdbl, B, nullptr, slot, nullptr, B, ssm_pool, S, L.g, L.status,
                            nullptr);
    sa.w_dt = w->dt_proj_w;
    // dt_proj fused into the state step (one launch, no dt round trip) when its rows allow
    hipError_t fused;
    {
        KernelTimer kt("decode.dt_proj_state", s);
        fused = launch_decode_dt_ssm(sa, adt == SSM_BF16, s);
    }
    if (fused != hipErrorNotSupported) {
        if (fused != hipSuccess) return hip_fail(fused, "decode.dt_proj_state");
    } else {
        SSM_TRY(gemm(B, E, R, xdbl, W, SSM_F32, w->dt_proj_w, R, adt, L.dt, E, adt, s, "decode.dt_proj", kGemmDtProj));
        SSM_TIMED("decode.state_update", s, launch_decode_ssm(sa, adt == SSM_BF16, s));
    }
    SSM_TRY(gemm(B, dm, E, L.g, E, adt, w->out_proj_w, E, adt, y, dm, adt, s, "decode.out_proj", kGemmOutProj,
                 L.splitk));
    return SSM_OK;
}

int prefill_checks(const ssm_shard_desc_t* d, const ssm_shard_weights_t* w, int64_t T, const ssm_seq_meta_t* m,
                   int32_t S, void* ws, size_t ws_bytes, PrefillWs* L) {
    SSM_TRY(common_checks(d, w, T, S));
    SSM_TRY(check_meta(m, T));
    *L = prefill_layout(d, T, m->nseq, nullptr);
    SSM_TRY(check_ws(ws, ws_bytes, L->total));
    *L = prefill_layout(d, T, m->nseq, ws);
    return SSM_OK;
}

int decode_checks(const ssm_shard_desc_t* d, const ssm_shard_weights_t* w, int32_t B, const int32_t* slot, int32_t S,
                  void* ws, size_t ws_bytes, DecodeWs* L) {
    SSM_TRY(common_checks(d, w, B, S));
    if (B < 0) return fail(SSM_E_INVAL, "batch %d", B);
    if (B > 0 && !slot) return fail(SSM_E_INVAL, "cache_slot is null");
    *L = decode_layout(d, B, nullptr);
    SSM_TRY(check_ws(ws, ws_bytes, L->total));
    *L = decode_layout(d, B, ws);
    return SSM_OK;
}

// ------------------------------------------------- decode step without allocation
// The decode workspace (status word, xz, u, x_dbl, dt, g, split-K partials) of
// ssm_shard_decode_step_noalloc lives in this file-scope device array. Every GPU the
// library runs on holds its own copy, at its own address, until the process ends. In host
// code `scratch` names a host-side stand-in, not device memory: its device address comes
// from hipGetSymbolAddress, once per device, and only that address is handed to kernels.
static __device__ __align__(256) char scratch[SSM_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::atomic<void*> g_scratch_dev[kMaxDevices];
std::mutex g_scratch_mu;

// device address of `scratch` on the device the launch goes to (looked up on the first
// call on that device, with that device current)
int scratch_address(hipStream_t s, void** out) {
    int dev = 0;
    SSM_TRY_HIP(hipGetDevice(&dev), "hipGetDevice");
    if (s) {
        hipDevice_t sdev = 0;
        SSM_TRY_HIP(hipStreamGetDevice(s, &sdev), "hipStreamGetDevice");
        if ((int)sdev != dev)
            return fail(SSM_E_INVAL, "the stream belongs to device %d but device %d is current", (int)sdev, dev);
    }
    if (dev < 0 || dev >= kMaxDevices) return fail(SSM_E_INVAL, "device %d: at most %d devices", dev, kMaxDevices);
    void* p = g_scratch_dev[dev].load(std::memory_order_acquire);
    if (!p) {
        std::lock_guard<std::mutex> lock(g_scratch_mu);
        p = g_scratch_dev[dev].load(std::memory_order_relaxed);
        if (!p) {
            SSM_TRY_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)), "hipGetSymbolAddress(scratch)");
            if (!p) return fail(SSM_E_HIP, "hipGetSymbolAddress(scratch) returned null");
            g_scratch_dev[dev].store(p, std::memory_order_release);
        }
    }
    *out = p;
    return SSM_OK;
}

}  // namespace

// ======================================================================= C ABI
extern "C" {

int ssm_shard_abi_version(void) { return SSM_SHARD_ABI_VERSION; }

const char* ssm_last_error(void) { return g_err.c_str(); }

int ssm_shard_check_desc(const ssm_shard_desc_t* desc) { return check_desc(desc); }

int ssm_shard_check_meta_host(const int32_t* cu, const int32_t* slot, const int32_t* hi, int32_t nseq, int64_t T,
                              int32_t num_slots) {
    if (nseq < 0) return fail(SSM_E_INVAL, "nseq %d", nseq);
    if (nseq == 0) return T == 0 ? SSM_OK : fail(SSM_E_SEQLENS, "T = %lld tokens but no sequences", (long long)T);
    if (!cu || !slot || !hi) return fail(SSM_E_INVAL, "metadata arrays must be non-null");
    if (cu[0] != 0) return fail(SSM_E_SEQLENS, "cu_seqlens[0] = %d, expected 0", cu[0]);
    for (int i = 0; i < nseq; ++i)
        if (cu[i + 1] < cu[i]) return fail(SSM_E_SEQLENS, "cu_seqlens decreases at %d", i + 1);
    if ((int64_t)cu[nseq] != T) return fail(SSM_E_SEQLENS, "cu_seqlens[nseq] = %d, expected T = %lld", cu[nseq], (long long)T);
    if (num_slots <= 0) return fail(SSM_E_INVAL, "num_slots %d", num_slots);
    std::vector<char> seen((size_t)num_slots, 0);
    for (int i = 0; i < nseq; ++i) {
        if (slot[i] < 0 || slot[i] >= num_slots) return fail(SSM_E_SLOT, "cache_slot[%d] = %d not in [0, %d)", i, slot[i], num_slots);
        if (seen[(size_t)slot[i]]) return fail(SSM_E_SLOT, "cache_slot %d used twice", slot[i]);
        seen[(size_t)slot[i]] = 1;
        if (hi[i] != 0 && hi[i] != 1) return fail(SSM_E_INVAL, "has_initial_state[%d] = %d", i, hi[i]);
    }
    return SSM_OK;
}

int ssm_shard_prefill_workspace_bytes(const ssm_shard_desc_t* desc, int64_t max_tokens, int32_t max_seqs, size_t* bytes) {
    SSM_TRY(check_desc(desc));
    if (!bytes || max_tokens < 0 || max_tokens > INT32_MAX || max_seqs < 0) return fail(SSM_E_INVAL, "bad size query");
    *bytes = prefill_layout(desc, max_tokens, max_seqs, nullptr).total;
    return SSM_OK;
}

int ssm_shard_decode_workspace_bytes(const ssm_shard_desc_t* desc, int32_t max_batch, size_t* bytes) {
    SSM_TRY(check_desc(desc));
    if (!bytes || max_batch < 0) return fail(SSM_E_INVAL, "bad size query");
    *bytes = decode_layout(desc, max_batch, nullptr).total;
    return SSM_OK;
}

int ssm_shard_workspace_init(void* ws, size_t ws_bytes, hipStream_t stream) {
    SSM_TRY(check_ws(ws, ws_bytes, kWsHeader));
    SSM_TRY_HIP(launch_fill_zero(ws, kWsHeader, stream), "workspace init");
    return SSM_OK;
}

int ssm_shard_take_status(void* ws, size_t ws_bytes, int32_t* status, hipStream_t stream) {
    SSM_TRY(check_ws(ws, ws_bytes, kWsHeader));
    if (!status) return fail(SSM_E_INVAL, "status is null");
    SSM_TRY_HIP(hipStreamSynchronize(stream), "sync");
    SSM_TRY_HIP(hipMemcpy(status, ws, sizeof(int32_t), hipMemcpyDeviceToHost), "read status");
    SSM_TRY_HIP(launch_fill_zero(ws, kWsHeader, stream), "clear status");
    SSM_TRY_HIP(hipStreamSynchronize(stream), "sync");
    return SSM_OK;
}

int ssm_shard_prefill_stage1(const ssm_shard_desc_t* d, const ssm_shard_weights_t* w, const void* x, int64_t T,
                             const ssm_seq_meta_t* m, void* conv_pool, int32_t S, float* xdbl, void* ws,
                             size_t ws_bytes, hipStream_t s) {
    PrefillWs L;
    SSM_TRY(prefill_checks(d, w, T, m, S, ws, ws_bytes, &L));
    if (d->d_conv > 1) SSM_TRY(check_ptr(conv_pool, "conv_pool"));  // K = 1 keeps no history
    if (T > 0) {
        SSM_TRY(check_ptr(x, "x"));
        SSM_TRY(check_ptr(xdbl, "x_dbl_partial"));
    }
    return prefill1(d, w, x, T, m, conv_pool, S, xdbl, L, s);
}

int ssm_shard_prefill_stage2(const ssm_shard_desc_t* d, const ssm_shard_weights_t* w, const float* xdbl, int64_t T,
                             const ssm_seq_meta_t* m, float* ssm_pool, int32_t S, void* y, void* ws, size_t ws_bytes,
                             hipStream_t s) {
    PrefillWs L;
    SSM_TRY(prefill_checks(d, w, T, m, S, ws, ws_bytes, &L));
    SSM_TRY(check_ptr(ssm_pool, "ssm_pool"));
    if (T > 0) {
        SSM_TRY(check_ptr(xdbl, "x_dbl"));
        SSM_TRY(check_ptr(y, "y_partial"));
    }
    return prefill2(d, w, xdbl, T, m, ssm_pool, S, y, L, s);
}

int ssm_shard_prefill(const ssm_shard_desc_t* d, const ssm_shard_weights_t* w, const void* x, int64_t T,
                      const ssm_seq_meta_t* m, void* conv_pool, float* ssm_pool, int32_t S, void* y, void* ws,
                      size_t ws_bytes, hipStream_t s) {
    PrefillWs L;
    SSM_TRY(prefill_checks(d, w, T, m, S, ws, ws_bytes, &L));
    if (d->d_conv > 1) SSM_TRY(check_ptr(conv_pool, "conv_pool"));  // K = 1 keeps no history
    SSM_TRY(check_ptr(ssm_pool, "ssm_pool"));
    if (T > 0) {
        SSM_TRY(check_ptr(x, "x"));
        SSM_TRY(check_ptr(y, "y_partial"));
    }
    SSM_TRY(prefill1(d, w, x, T, m, conv_pool, S, L.xdbl, L, s));
    return prefill2(d, w, L.xdbl, T, m, ssm_pool, S, y, L, s);
}

int ssm_shard_decode_stage1(const ssm_shard_desc_t* d, const ssm_shard_weights_t* w, const void* x, int32_t B,
                            const int32_t* slot, void* conv_pool, int32_t S, float* xdbl, void* ws, size_t ws_bytes,
                            hipStream_t s) {
    DecodeWs L;
    SSM_TRY(decode_checks(d, w, B, slot, S, ws, ws_bytes, &L));
    if (d->d_conv > 1) SSM_TRY(check_ptr(conv_pool, "conv_pool"));  // K = 1 keeps no history
    if (B > 0) {
        SSM_TRY(check_ptr(x, "x_t"));
        SSM_TRY(check_ptr(xdbl, "x_dbl_partial"));
    }
    return decode1(d, w, x, B, slot, conv_pool, S, xdbl, L, s);
}

int ssm_shard_decode_stage2(const ssm_shard_desc_t* d, const ssm_shard_weights_t* w, const float* xdbl, int32_t B,
                            const int32_t* slot, float* ssm_pool, int32_t S, void* y, void* ws, size_t ws_bytes,
                            hipStream_t s) {
    DecodeWs L;
    SSM_TRY(decode_checks(d, w, B, slot, S, ws, ws_bytes, &L));
    SSM_TRY(check_ptr(ssm_pool, "ssm_pool"));
    if (B > 0) {
        SSM_TRY(check_ptr(xdbl, "x_dbl"));
        SSM_TRY(check_ptr(y, "y_partial"));
    }
    return decode2(d, w, xdbl, B, slot, ssm_pool, S, y, L, s);
}

int ssm_shard_decode_step(const ssm_shard_desc_t* d, const ssm_shard_weights_t* w, const void* x, int32_t B,
                          const int32_t* slot, void* conv_pool, float* ssm_pool, int32_t S, void* y, void* ws,
                          size_t ws_bytes, hipStream_t s) {
    DecodeWs L;
    SSM_TRY(decode_checks(d, w, B, slot, S, ws, ws_bytes, &L));
    if (d->d_conv > 1) SSM_TRY(check_ptr(conv_pool, "conv_pool"));  // K = 1 keeps no history
    SSM_TRY(check_ptr(ssm_pool, "ssm_pool"));
    if (B > 0) {
        SSM_TRY(check_ptr(x, "x_t"));
        SSM_TRY(check_ptr(y, "y_partial"));
    }
    SSM_TRY(decode1(d, w, x, B, slot, conv_pool, S, L.xdbl, L, s));
    return decode2(d, w, L.xdbl, B, slot, ssm_pool, S, y, L, s);
}

int ssm_shard_decode_step_noalloc(const ssm_shard_desc_t* d, const ssm_shard_weights_t* w, const void* x,
                                  int32_t B, const int32_t* slot, void* conv_pool, float* ssm_pool, int32_t S,
                                  void* y, hipStream_t s) {
    SSM_TRY(common_checks(d, w, B, S));
    if (B < 0) return fail(SSM_E_INVAL, "batch %d", B);
    if (B > 0 && !slot) return fail(SSM_E_INVAL, "cache_slot is null");
    const size_t need = decode_layout(d, B, nullptr).total;
    if (need > (size_t)SSM_NOALLOC_SCRATCH_BYTES)
        return fail(SSM_E_WORKSPACE,
                    "a decode step of %d sequences needs %zu bytes of scratch; the static scratch holds %zu "
                    "(use ssm_shard_decode_step with a workspace)",
                    B, need, (size_t)SSM_NOALLOC_SCRATCH_BYTES);
    if (d->d_conv > 1) SSM_TRY(check_ptr(conv_pool, "conv_pool"));  // K = 1 keeps no history
    SSM_TRY(check_ptr(ssm_pool, "ssm_pool"));
    if (B > 0) {
        SSM_TRY(check_ptr(x, "x_t"));
        SSM_TRY(check_ptr(y, "y_partial"));
    }
    void* base = nullptr;
    SSM_TRY(scratch_address(s, &base));
    const DecodeWs L = decode_layout(d, B, base);
    SSM_TRY(decode1(d, w, x, B, slot, conv_pool, S, L.xdbl, L, s));
    return decode2(d, w, L.xdbl, B, slot, ssm_pool, S, y, L, s);
}

int ssm_shard_slice_weights(const ssm_shard_desc_t* d, const ssm_shard_weights_t* full, const ssm_shard_weights_t* out,
                            hipStream_t s) {
    SSM_TRY(check_desc(d));
    SSM_TRY(check_weights(full));
    SSM_TRY(check_weights(out));
    const size_t a = act_bytes(d);
    const int64_t E = d->d_inner_shard, Et = d->d_inner_total, c0 = (int64_t)d->shard_index * E;
    const int64_t dm = d->d_model, K = d->d_conv, R = d->dt_rank, N = d->d_state, W = R + 2 * N;
    auto cp = [&](const void* src, int64_t ld_src, void* dst, int64_t ld_dst, int64_t rows, int64_t row_bytes,
                  const char* what) -> int {
        SSM_TRY_HIP(launch_copy_rows(dst, ld_dst, src, ld_src, rows, row_bytes, s), what);
        return SSM_OK;
    };
    const char* fin = (const char*)full->in_proj_w;
    SSM_TRY(cp(fin + c0 * dm * a, dm * a, (void*)out->in_proj_w, dm * a, E, dm * a, "slice in_proj x rows"));
    SSM_TRY(cp(fin + (Et + c0) * dm * a, dm * a, (char*)out->in_proj_w + E * dm * a, dm * a, E, dm * a,
               "slice in_proj z rows"));
    SSM_TRY(cp((const char*)full->conv_w + c0 * K * a, E * K * a, (void*)out->conv_w, E * K * a, 1, E * K * a, "slice conv_w"));
    SSM_TRY(cp((const char*)full->conv_b + c0 * a, E * a, (void*)out->conv_b, E * a, 1, E * a, "slice conv_b"));
    SSM_TRY(cp((const char*)full->x_proj_w + c0 * a, Et * a, (void*)out->x_proj_w, E * a, W, E * a, "slice x_proj"));
    SSM_TRY(cp((const char*)full->dt_proj_w + c0 * R * a, E * R * a, (void*)out->dt_proj_w, E * R * a, 1, E * R * a,
               "slice dt_proj"));
    SSM_TRY(cp((const char*)full->out_proj_w + c0 * a, Et * a, (void*)out->out_proj_w, E * a, dm, E * a, "slice out_proj"));
    SSM_TRY(cp((const char*)full->dt_proj_b + c0 * 4, E * 4, (void*)out->dt_proj_b, E * 4, 1, E * 4, "slice dt_proj_b"));
    SSM_TRY(cp((const char*)full->A_log + c0 * N * 4, E * N * 4, (void*)out->A_log, E * N * 4, 1, E * N * 4, "slice A_log"));
    SSM_TRY(cp((const char*)full->D + c0 * 4, E * 4, (void*)out->D, E * 4, 1, E * 4, "slice D"));
    return SSM_OK;
}

int ssm_reduce_add_f32(float* dst, const float* src, int64_t n, hipStream_t s) {
    if (n < 0) return fail(SSM_E_INVAL, "n %lld", (long long)n);
    if (n == 0) return SSM_OK;
    SSM_TRY(check_ptr(dst, "dst"));
    SSM_TRY(check_ptr(src, "src"));
    SSM_TIMED("exchange.reduce_add", s, launch_reduce_add(dst, src, n, s));
    return SSM_OK;
}

namespace {
const char* const kCodecEncodeName[] = {"exchange.encode_f16", "exchange.encode_bf16", "exchange.encode_fp8",
                                        "exchange.encode_int8"};
const char* const kCodecDecodeName[] = {"exchange.decode_f16", "exchange.decode_bf16", "exchange.decode_fp8",
                                        "exchange.decode_int8"};

int check_codec_shape(int32_t codec, int64_t rows, int64_t cols) {
    if (codec < SSM_CODEC_F16 || codec > SSM_CODEC_INT8) return fail(SSM_E_INVAL, "codec %d", codec);
    if (rows < 0 || cols < 0) return fail(SSM_E_INVAL, "payload shape %lld x %lld", (long long)rows, (long long)cols);
    if (cols % 8 != 0) return fail(SSM_E_ALIGN, "cols %lld is not a multiple of 8", (long long)cols);
    return SSM_OK;
}
}  // namespace

int ssm_exchange_payload_bytes(int32_t codec, int64_t rows, int64_t cols, size_t* bytes) {
    SSM_TRY(check_codec_shape(codec, rows, cols));
    if (!bytes) return fail(SSM_E_INVAL, "bytes is null");
    *bytes = codec_payload_bytes(codec, rows, cols);
    return SSM_OK;
}

int ssm_exchange_encode(int32_t codec, const void* src, int32_t src_dtype, int64_t rows, int64_t cols, int64_t ld_src,
                        void* payload, size_t payload_bytes, hipStream_t s) {
    SSM_TRY(check_codec_shape(codec, rows, cols));
    if (src_dtype != SSM_F32 && src_dtype != SSM_BF16) return fail(SSM_E_INVAL, "src_dtype %d", src_dtype);
    if (rows == 0 || cols == 0) return SSM_OK;
    if (ld_src < cols) return fail(SSM_E_INVAL, "ld_src %lld < cols %lld", (long long)ld_src, (long long)cols);
    if (ld_src % 8 != 0) return fail(SSM_E_ALIGN, "ld_src %lld is not a multiple of 8", (long long)ld_src);
    SSM_TRY(check_ptr(src, "src"));
    SSM_TRY(check_ptr(payload, "payload"));
    if (payload_bytes < codec_payload_bytes(codec, rows, cols))
        return fail(SSM_E_WORKSPACE, "payload %zu bytes < %zu needed", payload_bytes, codec_payload_bytes(codec, rows, cols));
    SSM_TIMED(kCodecEncodeName[codec], s, launch_codec_encode(codec, src, src_dtype == SSM_BF16, ld_src, rows, cols, payload, s));
    return SSM_OK;
}

int ssm_exchange_decode_accumulate(int32_t codec, const void* payload, size_t payload_bytes, int64_t rows, int64_t cols,
                                   float* acc, int64_t ld_acc, int32_t accumulate, hipStream_t s) {
    SSM_TRY(check_codec_shape(codec, rows, cols));
    if (rows == 0 || cols == 0) return SSM_OK;
    if (ld_acc < cols) return fail(SSM_E_INVAL, "ld_acc %lld < cols %lld", (long long)ld_acc, (long long)cols);
    if (ld_acc % 8 != 0) return fail(SSM_E_ALIGN, "ld_acc %lld is not a multiple of 8", (long long)ld_acc);
    SSM_TRY(check_ptr(payload, "payload"));
    SSM_TRY(check_ptr(acc, "acc"));
    if (payload_bytes < codec_payload_bytes(codec, rows, cols))
        return fail(SSM_E_WORKSPACE, "payload %zu bytes < %zu needed", payload_bytes, codec_payload_bytes(codec, rows, cols));
    SSM_TIMED(kCodecDecodeName[codec], s,
              launch_codec_decode_acc(codec, payload, rows, cols, acc, ld_acc, accumulate != 0, s));
    return SSM_OK;
}

int ssm_gemm_nt(int64_t M, int64_t N, int64_t K, const void* A, int64_t lda, int32_t adt, const void* B, int64_t ldb,
                int32_t bdt, void* C, int64_t ldc, int32_t cdt, hipStream_t s) {
    if (M < 0 || N < 0 || K < 0 || M > INT32_MAX || N > INT32_MAX || K > INT32_MAX)
        return fail(SSM_E_INVAL, "gemm size %lld x %lld x %lld", (long long)M, (long long)N, (long long)K);
    for (int32_t dt : {adt, bdt, cdt})
        if (dt != SSM_F32 && dt != SSM_BF16) return fail(SSM_E_INVAL, "dtype %d", dt);
    if (bdt == SSM_F32 && (adt != SSM_F32 || cdt != SSM_F32))
        return fail(SSM_E_INVAL, "float32 B needs float32 A and C");
    if (M == 0 || N == 0) return SSM_OK;
    if (K % 8 || lda % 8 || ldb % 8 || ldc % 4) return fail(SSM_E_ALIGN, "K, lda, ldb must be multiples of 8, ldc of 4");
    if (lda < K || ldb < K || ldc < N) return fail(SSM_E_INVAL, "leading dimension smaller than the row");
    SSM_TRY(check_ptr(A, "A"));
    SSM_TRY(check_ptr(B, "B"));
    SSM_TRY(check_ptr(C, "C"));
    return gemm(M, N, K, A, lda, adt, B, ldb, bdt, C, ldc, cdt, s, "op.gemm");
}

int ssm_gemm_splitk_bytes(int64_t M, int64_t N, int64_t K, int32_t adt, int32_t bdt, int32_t role, size_t* bytes) {
    if (!bytes || M < 0 || N < 0 || K < 0 || role < kGemmGeneric || role > kGemmOutProj)
        return fail(SSM_E_INVAL, "bad split-K size query");
    *bytes = gemm_splitk_bytes(M, N, K, adt, bdt, (GemmRole)role);
    return SSM_OK;
}

int ssm_gemm_nt_role(int64_t M, int64_t N, int64_t K, const void* A, int64_t lda, int32_t adt, const void* B,
                     int64_t ldb, int32_t bdt, void* C, int64_t ldc, int32_t cdt, int32_t role, float* scratch,
                     size_t scratch_bytes, hipStream_t s) {
    if (role < kGemmGeneric || role > kGemmOutProj) return fail(SSM_E_INVAL, "gemm role %d", role);
    if (scratch_bytes > 0) SSM_TRY(check_ptr(scratch, "scratch"));
    if (M < 0 || N < 0 || K < 0 || M > INT32_MAX || N > INT32_MAX || K > INT32_MAX)
        return fail(SSM_E_INVAL, "gemm size %lld x %lld x %lld", (long long)M, (long long)N, (long long)K);
    for (int32_t dt : {adt, bdt, cdt})
        if (dt != SSM_F32 && dt != SSM_BF16) return fail(SSM_E_INVAL, "dtype %d", dt);
    if (bdt == SSM_F32 && (adt != SSM_F32 || cdt != SSM_F32))
        return fail(SSM_E_INVAL, "float32 B needs float32 A and C");
    if (M == 0 || N == 0) return SSM_OK;
    if (K % 8 || lda % 8 || ldb % 8 || ldc % 4) return fail(SSM_E_ALIGN, "K, lda, ldb must be multiples of 8, ldc of 4");
    if (lda < K || ldb < K || ldc < N) return fail(SSM_E_INVAL, "leading dimension smaller than the row");
    SSM_TRY(check_ptr(A, "A"));
    SSM_TRY(check_ptr(B, "B"));
    SSM_TRY(check_ptr(C, "C"));
    Scratch sk;
    sk.p = scratch;
    sk.bytes = scratch ? scratch_bytes : 0;
    return gemm(M, N, K, A, lda, adt, B, ldb, bdt, C, ldc, cdt, s, "op.gemm", (GemmRole)role, sk);
}

int ssm_conv1d_silu(const ssm_shard_desc_t* d, const ssm_shard_weights_t* w, const void* xz, int64_t T,
                    const ssm_seq_meta_t* m, void* conv_pool, int32_t S, void* u, void* ws, size_t ws_bytes,
                    hipStream_t s) {
    SSM_TRY(common_checks(d, w, T, S));
    SSM_TRY(check_meta(m, T));
    SSM_TRY(check_ws(ws, ws_bytes, kWsHeader));
    if (d->d_conv > 1) SSM_TRY(check_ptr(conv_pool, "conv_pool"));  // K = 1 keeps no history
    if (T > 0) {
        SSM_TRY(check_ptr(xz, "xz"));
        SSM_TRY(check_ptr(u, "u"));
    }
    ConvArgs ca = conv_args(d, w, xz, T, m->cu_seqlens, m->cache_slot, m->has_initial_state, m->nseq, conv_pool, S, u,
                            (int32_t*)ws);
    SSM_TIMED("op.conv1d", s, launch_conv_prefill(ca, d->act_dtype == SSM_BF16, s));
    SSM_TIMED("op.conv_history", s, launch_conv_state_update(ca, d->act_dtype == SSM_BF16, s));
    return SSM_OK;
}

int ssm_selective_scan(const ssm_shard_desc_t* d, const ssm_shard_weights_t* w, const void* u, const void* dt,
                       const void* xz, const float* xdbl, int64_t T, const ssm_seq_meta_t* m, float* pool, int32_t S,
                       void* g, void* ws, size_t ws_bytes, hipStream_t s) {
    SSM_TRY(common_checks(d, w, T, S));
    SSM_TRY(check_meta(m, T));
    const size_t need = kWsHeader + scan_scratch_bytes(T, d->d_inner_shard, m->nseq);
    SSM_TRY(check_ws(ws, ws_bytes, need));
    SSM_TRY(check_ptr(pool, "ssm_pool"));
    if (T > 0) {
        SSM_TRY(check_ptr(u, "u"));
        SSM_TRY(check_ptr(dt, "dt"));
        SSM_TRY(check_ptr(xz, "xz"));
        SSM_TRY(check_ptr(xdbl, "x_dbl"));
        SSM_TRY(check_ptr(g, "g"));
    }
    ScanArgs sa = scan_args(d, w, u, dt, xz, xdbl, T, m->cu_seqlens, m->cache_slot, m->has_initial_state, m->nseq,
                            pool, S, g, (int32_t*)ws, (char*)ws + kWsHeader);
    SSM_TRY_HIP(launch_scan_prefill(sa, d->act_dtype == SSM_BF16, s), "selective scan");
    return SSM_OK;
}

int ssm_decode_conv(const ssm_shard_desc_t* d, const ssm_shard_weights_t* w, const void* xz, int32_t B,
                    const int32_t* slot, void* conv_pool, int32_t S, void* u, void* ws, size_t ws_bytes,
                    hipStream_t s) {
    SSM_TRY(common_checks(d, w, B, S));
    SSM_TRY(check_ws(ws, ws_bytes, kWsHeader));
    if (d->d_conv > 1) SSM_TRY(check_ptr(conv_pool, "conv_pool"));  // K = 1 keeps no history
    if (B < 0) return fail(SSM_E_INVAL, "batch %d", B);
    if (B > 0) {
        if (!slot) return fail(SSM_E_INVAL, "cache_slot is null");
        SSM_TRY(check_ptr(xz, "xz"));
        SSM_TRY(check_ptr(u, "u"));
    }
    ConvArgs ca = conv_args(d, w, xz, B, nullptr, slot, nullptr, B, conv_pool, S, u, (int32_t*)ws);
    SSM_TIMED("op.decode_conv", s, launch_conv_decode(ca, d->act_dtype == SSM_BF16, s));
    return SSM_OK;
}

int ssm_decode_ssm(const ssm_shard_desc_t* d, const ssm_shard_weights_t* w, const void* u, const void* dt,
                   const void* xz, const float* xdbl, int32_t B, const int32_t* slot, float* pool, int32_t S, void* g,
                   void* ws, size_t ws_bytes, hipStream_t s) {
    SSM_TRY(common_checks(d, w, B, S));
    SSM_TRY(check_ws(ws, ws_bytes, kWsHeader));
    SSM_TRY(check_ptr(pool, "ssm_pool"));
    if (B < 0) return fail(SSM_E_INVAL, "batch %d", B);
    if (B > 0) {
        if (!slot) return fail(SSM_E_INVAL, "cache_slot is null");
        SSM_TRY(check_ptr(u, "u"));
        SSM_TRY(check_ptr(dt, "dt"));
        SSM_TRY(check_ptr(xz, "xz"));
        SSM_TRY(check_ptr(xdbl, "x_dbl"));
        SSM_TRY(check_ptr(g, "g"));
    }
    ScanArgs sa = scan_args(d, w, u, dt, xz, xdbl, B, nullptr, slot, nullptr, B, pool, S, g, (int32_t*)ws, nullptr);
    SSM_TIMED("op.decode_state_update", s, launch_decode_ssm(sa, d->act_dtype == SSM_BF16, s));
    return SSM_OK;
}

}  // extern "C"

// ==================================================================== Mamba-2 (SSD) shard
// Prefill stage 1: in_proj GEMM -> [z | x | B | C | dt]; conv1d+SiLU over [x | B | C]
// (and the conv history); SSD passes -> g and final states; per-head sums of g^2 summed
// into norm groups. [exchange of the sums of squares: the caller's.] Stage 2: gated RMS
// normalisation -> out_proj GEMM. Decode: skinny in_proj, one conv step, one state step.
namespace {

struct M2 {
    int64_t dm, Etot, E, H, P, N, G, Gs, Cc, rows, K, r;
    int hpg, gsize, g_off;
    bool split;
};

int m2_dims(const ssm2_shard_desc_t* d, M2* o) {
    if (!d) return fail(SSM_E_INVAL, "desc is null");
    if (d->act_dtype != SSM_BF16) return fail(SSM_E_INVAL, "the Mamba-2 shard runs with bf16 activations");
    if (d->headdim != 64 || d->d_state != 128) return fail(SSM_E_INVAL, "headdim %d / d_state %d: 64 / 128 required", d->headdim, d->d_state);
    if (d->d_model <= 0 || d->d_model % 16) return fail(SSM_E_INVAL, "d_model %d must be a positive multiple of 16", d->d_model);
    if (d->shard_count <= 0 || d->shard_index < 0 || d->shard_index >= d->shard_count)
        return fail(SSM_E_INVAL, "shard %d of %d", d->shard_index, d->shard_count);
    if (d->ngroups_total <= 0 || d->nheads_total <= 0 || d->nheads_total % d->ngroups_total)
        return fail(SSM_E_INVAL, "nheads %d must be a positive multiple of ngroups %d", d->nheads_total, d->ngroups_total);
    if (d->nheads_total % d->shard_count) return fail(SSM_E_INVAL, "nheads %d not divisible by %d shards", d->nheads_total, d->shard_count);
    if (d->d_conv < 2 || d->d_conv > kMaxConv) return fail(SSM_E_INVAL, "d_conv %d not in [2, %d]", d->d_conv, kMaxConv);
    M2 m{};
    m.dm = d->d_model; m.P = 64; m.N = 128; m.G = d->ngroups_total; m.K = d->d_conv; m.r = d->shard_index;
    m.H = d->nheads_total / d->shard_count;
    if (m.H % 8) return fail(SSM_E_INVAL, "%lld heads per shard: a multiple of 8 is required", (long long)m.H);
    m.E = m.H * m.P; m.Etot = (int64_t)d->nheads_total * m.P;
    m.split = m.G % d->shard_count == 0;
    m.Gs = m.split ? m.G / d->shard_count : m.G;
    m.Cc = m.E + 2 * m.Gs * m.N;
    m.rows = 2 * m.E + 2 * m.Gs * m.N + m.H;
    m.hpg = (int)(d->nheads_total / m.G);
    m.gsize = (int)(m.Etot / m.G);
    m.g_off = m.split ? (int)(m.r * m.Gs) : 0;
    *o = m;
    return SSM_OK;
}

int m2_check_weights(const ssm2_shard_weights_t* w) {
    if (!w) return fail(SSM_E_INVAL, "weights is null");
    const void* ps[] = {w->in_proj_w, w->conv_w, w->conv_b, w->out_proj_w, w->dt_bias, w->A_log, w->D, w->norm_w};
    const char* names[] = {"in_proj_w", "conv_w", "conv_b", "out_proj_w", "dt_bias", "A_log", "D", "norm_w"};
    for (int i = 0; i < 8; ++i) {
        if (!ps[i]) return fail(SSM_E_INVAL, "weights.%s is null", names[i]);
        if (!aligned16(ps[i])) return fail(SSM_E_ALIGN, "weights.%s is not 16-byte aligned", names[i]);
    }
    return SSM_OK;
}

struct M2Ws {
    int32_t* status;
    char *zx, *u, *g, *gn;
    float* hs;
    char* plan;
    int32_t* count;
    float *states, *lsum;
    int win, maxw;
    Scratch splitk;
    size_t total;
};

M2Ws m2_layout(const M2& m, int64_t T, int nseq, bool prefill, void* base) {
    M2Ws L{};
    char* b = (char*)base;
    size_t off = kWsHeader;
    auto take = [&](size_t bytes) { char* p = b ? b + off : nullptr; off += align256(bytes); return p; };
    L.status = (int32_t*)b;
    L.zx = take((size_t)T * m.rows * 2);
    L.u = take((size_t)T * m.Cc * 2);
    L.g = take((size_t)T * m.E * 2);
    L.gn = take((size_t)T * m.E * 2);
    L.hs = (float*)take((size_t)T * m.H * 4);
    if (prefill) {
        L.win = ssd_window_len(T, (int)m.H);
        L.maxw = ssd_max_windows(T, nseq, L.win);
        L.plan = take((size_t)L.maxw * 16);
        L.count = (int32_t*)take(16);
        L.states = (float*)take(ssd_state_bytes(L.maxw, (int)m.H));
        L.lsum = (float*)take((size_t)L.maxw * m.H * 4);
    }
    const size_t sk = std::max(gemm_splitk_bytes(T, m.rows, m.dm, SSM_BF16, SSM_BF16, kGemmInProj),
                               gemm_splitk_bytes(T, m.dm, m.E, SSM_BF16, SSM_BF16, kGemmOutProj));
    L.splitk.p = (float*)take(sk);
    L.splitk.bytes = sk;
    L.total = off;
    return L;
}

SsdPublic m2_ssd(const M2& m, const ssm2_shard_weights_t* w, const M2Ws& L, float* pool, int S, int32_t* status) {
    SsdPublic p{};
    p.zx = L.zx; p.ld_zx = m.rows; p.u = L.u; p.ld_u = m.Cc;
    p.dt_col = (int)(2 * m.E + 2 * m.Gs * m.N); p.b_col = (int)m.E; p.c_col = (int)(m.E + m.Gs * m.N);
    p.H = (int)m.H; p.h_global0 = (int)(m.r * m.H); p.hpg = m.hpg; p.g_off = m.g_off;
    p.dt_bias = w->dt_bias; p.A_log = w->A_log; p.D = w->D;
    p.g = L.g; p.hs = L.hs; p.pool = pool; p.S = S; p.status = status;
    return p;
}

ConvArgs m2_conv(const M2& m, const ssm2_shard_weights_t* w, const M2Ws& L, int64_t T, const int32_t* cu,
                 const int32_t* slot, const int32_t* hi, int nseq, void* conv_pool, int S) {
    ConvArgs a{};
    a.xz = L.zx + m.E * 2; a.ld_xz = m.rows;   // [x | B | C] columns of the in_proj output
    a.w = w->conv_w; a.b = w->conv_b; a.u = L.u; a.conv_pool = conv_pool;
    a.cu = cu; a.slot = slot; a.has_init = hi; a.status = L.status;
    a.T = T; a.E = (int)m.Cc; a.K = (int)m.K; a.nseq = nseq; a.S = S;
    return a;
}

int m2_stage2(const M2& m, const ssm2_shard_weights_t* w, const float* sumsq, int64_t T, void* y, const M2Ws& L,
              hipStream_t s, const char* norm_name, const char* out_name, const char* fused_name = nullptr) {
    if (fused_name && T <= 16) {
        // a few rows (a decode step): the gated norm as the streamed out_proj's operand
        // transform, one launch instead of two
        SkinnyArgs p = skinny(L.g, m.E, false, w->out_proj_w, m.E, y, m.dm, T, m.dm, m.E);
        p.nrm_sumsq = sumsq; p.nrm_w = w->norm_w; p.nrm_G = (int)m.G; p.nrm_gsize = m.gsize;
        p.nrm_c0 = (int)(m.r * m.E); p.nrm_eps = 1e-5f;
        hipError_t e;
        {
            KernelTimer kt(fused_name, s);
            e = launch_gemv_norm(p, s);
        }
        if (e == hipSuccess) return SSM_OK;
        if (e != hipErrorNotSupported) return fail(SSM_E_HIP, "%s: %s", fused_name, hipGetErrorString(e));
    }
    SSM_TIMED(norm_name, s, launch_ssd_norm(L.g, sumsq, w->norm_w, L.gn, T, (int)m.E, (int)m.G, m.gsize,
                                            (int)(m.r * m.E), 1e-5f, s));
    return gemm(T, m.dm, m.E, L.gn, m.E, SSM_BF16, w->out_proj_w, m.E, SSM_BF16, y, m.dm, SSM_BF16, s, out_name,
                kGemmOutProj, L.splitk);
}

}  // namespace

extern "C" {

int ssm2_shard_check_desc(const ssm2_shard_desc_t* d) {
    M2 m;
    return m2_dims(d, &m);
}

int ssm2_shard_prefill_workspace_bytes(const ssm2_shard_desc_t* d, int64_t max_tokens, int32_t max_seqs, size_t* bytes) {
    M2 m;
    SSM_TRY(m2_dims(d, &m));
    if (!bytes) return fail(SSM_E_INVAL, "bytes is null");
    if (max_tokens < 0 || max_seqs < 0) return fail(SSM_E_INVAL, "negative size");
    *bytes = m2_layout(m, max_tokens, max_seqs, true, nullptr).total;
    return SSM_OK;
}

int ssm2_shard_decode_workspace_bytes(const ssm2_shard_desc_t* d, int32_t max_batch, size_t* bytes) {
    M2 m;
    SSM_TRY(m2_dims(d, &m));
    if (!bytes) return fail(SSM_E_INVAL, "bytes is null");
    if (max_batch < 0) return fail(SSM_E_INVAL, "negative size");
    *bytes = m2_layout(m, max_batch, 0, false, nullptr).total;
    return SSM_OK;
}

int ssm2_shard_slice_weights(const ssm2_shard_desc_t* d, const ssm2_shard_weights_t* full,
                             const ssm2_shard_weights_t* out, hipStream_t s) {
    M2 m;
    SSM_TRY(m2_dims(d, &m));
    SSM_TRY(m2_check_weights(full));
    SSM_TRY(m2_check_weights(out));
    const int64_t dm = m.dm, Et = m.Etot, E = m.E, N = m.N, G = m.G, Gs = m.Gs, H = m.H, K = m.K;
    const int64_t g0 = m.g_off, c0 = m.r * E, h0 = m.r * H;
    const int64_t rows_full = 2 * Et + 2 * G * N + (int64_t)(Et / m.P);
    (void)rows_full;
    auto cp = [&](const void* src, int64_t ld_src, void* dst, int64_t ld_dst, int64_t rows, int64_t row_bytes,
                  const char* what) -> int {
        SSM_TRY_HIP(launch_copy_rows(dst, ld_dst, src, ld_src, rows, row_bytes, s), what);
        return SSM_OK;
    };
    const char* fin = (const char*)full->in_proj_w;
    char* oin = (char*)out->in_proj_w;
    const int64_t rb = dm * 2;  // bytes per in_proj row
    SSM_TRY(cp(fin + c0 * rb, rb, oin, rb, E, rb, "slice z rows"));
    SSM_TRY(cp(fin + (Et + c0) * rb, rb, oin + E * rb, rb, E, rb, "slice x rows"));
    SSM_TRY(cp(fin + (2 * Et + g0 * N) * rb, rb, oin + 2 * E * rb, rb, Gs * N, rb, "slice B rows"));
    SSM_TRY(cp(fin + (2 * Et + G * N + g0 * N) * rb, rb, oin + (2 * E + Gs * N) * rb, rb, Gs * N, rb, "slice C rows"));
    SSM_TRY(cp(fin + (2 * Et + 2 * G * N + h0) * rb, rb, oin + (2 * E + 2 * Gs * N) * rb, rb, H, rb, "slice dt rows"));
    const char* fcw = (const char*)full->conv_w;
    char* ocw = (char*)out->conv_w;
    const int64_t cb = K * 2;
    SSM_TRY(cp(fcw + c0 * cb, cb, ocw, cb, E, cb, "slice conv x"));
    SSM_TRY(cp(fcw + (Et + g0 * N) * cb, cb, ocw + E * cb, cb, Gs * N, cb, "slice conv B"));
    SSM_TRY(cp(fcw + (Et + G * N + g0 * N) * cb, cb, ocw + (E + Gs * N) * cb, cb, Gs * N, cb, "slice conv C"));
    const char* fcb = (const char*)full->conv_b;
    char* ocb = (char*)out->conv_b;
    SSM_TRY(cp(fcb + c0 * 2, 2, ocb, 2, E, 2, "slice conv_b x"));
    SSM_TRY(cp(fcb + (Et + g0 * N) * 2, 2, ocb + E * 2, 2, Gs * N, 2, "slice conv_b B"));
    SSM_TRY(cp(fcb + (Et + G * N + g0 * N) * 2, 2, ocb + (E + Gs * N) * 2, 2, Gs * N, 2, "slice conv_b C"));
    SSM_TRY(cp(full->dt_bias + h0, 4, (void*)out->dt_bias, 4, H, 4, "slice dt_bias"));
    SSM_TRY(cp(full->A_log + h0, 4, (void*)out->A_log, 4, H, 4, "slice A_log"));
    SSM_TRY(cp(full->D + h0, 4, (void*)out->D, 4, H, 4, "slice D"));
    SSM_TRY(cp(full->norm_w + c0, 4, (void*)out->norm_w, 4, E, 4, "slice norm_w"));
    SSM_TRY(cp((const char*)full->out_proj_w + c0 * 2, Et * 2, (void*)out->out_proj_w, E * 2, dm, E * 2,
               "slice out_proj columns"));
    return SSM_OK;
}

int ssm2_shard_prefill_stage1(const ssm2_shard_desc_t* d, const ssm2_shard_weights_t* w, const void* x, int64_t T,
                              const ssm_seq_meta_t* meta, void* conv_pool, float* ssm_pool, int32_t S,
                              float* sumsq_partial, void* ws, size_t ws_bytes, hipStream_t s) {
    M2 m;
    SSM_TRY(m2_dims(d, &m));
    SSM_TRY(m2_check_weights(w));
    if (T < 0 || S <= 0) return fail(SSM_E_INVAL, "T %lld, num_slots %d", (long long)T, S);
    SSM_TRY(check_meta(meta, T));
    SSM_TRY(check_ptr(conv_pool, "conv_pool"));
    SSM_TRY(check_ptr(ssm_pool, "ssm_pool"));
    M2Ws L = m2_layout(m, T, meta->nseq, true, nullptr);
    SSM_TRY(check_ws(ws, ws_bytes, L.total));
    L = m2_layout(m, T, meta->nseq, true, ws);
    if (meta->nseq == 0) return SSM_OK;
    if (T > 0) {
        SSM_TRY(check_ptr(x, "x"));
        SSM_TRY(check_ptr(sumsq_partial, "sumsq_partial"));
        // [z ‖ x] and [B ‖ C ‖ dt] as two products: the 2E columns fill whole 256-wide tiles,
        // and the few others run on narrower tiles instead of a mostly empty last tile column
        // (for 16384 tokens of the 2.7B half shard: 5 rounds of tiles plus a small product,
        // where the 5416 columns at once took 6 rounds)
        const int64_t nzx = 2 * m.E, nbc = m.rows - nzx;
        SSM_TRY(gemm(T, nzx, m.dm, x, m.dm, SSM_BF16, w->in_proj_w, m.dm, SSM_BF16, L.zx, m.rows, SSM_BF16, s,
                     "m2.prefill.in_proj", kGemmInProj, L.splitk));
        SSM_TRY(gemm(T, nbc, m.dm, x, m.dm, SSM_BF16, (const char*)w->in_proj_w + nzx * m.dm * 2, m.dm, SSM_BF16,
                     L.zx + nzx * 2, m.rows, SSM_BF16, s, "m2.prefill.in_proj_bcdt", kGemmInProj, L.splitk));
    }
    // (the history update also runs for a batch of empty sequences: fresh ones end with zeros)
    ConvArgs ca = m2_conv(m, w, L, T, meta->cu_seqlens, meta->cache_slot, meta->has_initial_state, meta->nseq,
                          conv_pool, S);
    SSM_TIMED("m2.prefill.conv1d", s, launch_conv_prefill(ca, true, s));
    SSM_TIMED("m2.prefill.conv_history", s, launch_conv_state_update(ca, true, s));
    SsdPublic p = m2_ssd(m, w, L, ssm_pool, S, L.status);
    p.cu = meta->cu_seqlens; p.slot = meta->cache_slot; p.has_init = meta->has_initial_state; p.nseq = meta->nseq;
    p.win = L.win; p.T = T; p.plan = L.plan; p.plan_count = L.count; p.max_windows = L.maxw; p.states = L.states; p.lsum = L.lsum;
    SSM_TRY_HIP(launch_ssd_prefill(p, s), "ssd prefill");
    if (T > 0)
        SSM_TIMED("m2.prefill.group_sumsq", s, launch_ssd_group_sumsq(L.hs, (int)m.H, (int)(m.r * m.H), m.hpg, (int)m.G,
                                                                     sumsq_partial, T, s));
    return SSM_OK;
}

int ssm2_shard_prefill_stage2(const ssm2_shard_desc_t* d, const ssm2_shard_weights_t* w, const float* sumsq, int64_t T,
                              void* y, void* ws, size_t ws_bytes, hipStream_t s) {
    M2 m;
    SSM_TRY(m2_dims(d, &m));
    SSM_TRY(m2_check_weights(w));
    if (T < 0) return fail(SSM_E_INVAL, "T %lld", (long long)T);
    if (T == 0) return SSM_OK;
    SSM_TRY(check_ptr(sumsq, "sumsq"));
    SSM_TRY(check_ptr(y, "y_partial"));
    // the stage-1 part of the layout does not depend on the sequence count
    M2Ws L = m2_layout(m, T, 0, false, nullptr);
    SSM_TRY(check_ws(ws, ws_bytes, L.total));
    L = m2_layout(m, T, 0, false, ws);
    return m2_stage2(m, w, sumsq, T, y, L, s, "m2.prefill.norm", "m2.prefill.out_proj");
}

int ssm2_shard_decode_stage1(const ssm2_shard_desc_t* d, const ssm2_shard_weights_t* w, const void* x, int32_t B,
                             const int32_t* slot, void* conv_pool, float* ssm_pool, int32_t S, float* sumsq_partial,
                             void* ws, size_t ws_bytes, hipStream_t s) {
    M2 m;
    SSM_TRY(m2_dims(d, &m));
    SSM_TRY(m2_check_weights(w));
    if (B < 0 || S <= 0) return fail(SSM_E_INVAL, "batch %d, num_slots %d", B, S);
    M2Ws L = m2_layout(m, B, 0, false, nullptr);
    SSM_TRY(check_ws(ws, ws_bytes, L.total));
    L = m2_layout(m, B, 0, false, ws);
    if (B == 0) return SSM_OK;
    SSM_TRY(check_ptr(x, "x_t"));
    if (!slot) return fail(SSM_E_INVAL, "cache_slot is null");
    SSM_TRY(check_ptr(conv_pool, "conv_pool"));
    SSM_TRY(check_ptr(ssm_pool, "ssm_pool"));
    SSM_TRY(check_ptr(sumsq_partial, "sumsq_partial"));
    if (B <= kConvEpilogueMax) {
        // in_proj with the conv window shift + SiLU of the x, B, C columns in its epilogue
        SkinnyArgs p = skinny(x, m.dm, false, w->in_proj_w, m.dm, L.zx, m.rows, B, m.rows, m.dm);
        p.slot = slot; p.S = S; p.status = L.status;
        p.conv_w = w->conv_w; p.conv_b = w->conv_b; p.conv_pool = conv_pool; p.Kc = (int)m.K;
        p.conv_lo = (int)m.E; p.conv_n = (int)m.Cc; p.u = L.u;
        SSM_SKINNY("m2.decode.in_proj_conv", s, p, kSkinnyConv);
    } else {
        SSM_TRY(gemm(B, m.rows, m.dm, x, m.dm, SSM_BF16, w->in_proj_w, m.dm, SSM_BF16, L.zx, m.rows, SSM_BF16, s,
                     "m2.decode.in_proj", kGemmInProj, L.splitk));
        ConvArgs ca = m2_conv(m, w, L, B, nullptr, slot, nullptr, B, conv_pool, S);
        SSM_TIMED("m2.decode.conv", s, launch_conv_decode(ca, true, s));
    }
    SsdPublic p = m2_ssd(m, w, L, ssm_pool, S, L.status);
    p.slot = slot;
    SSM_TIMED("m2.decode.state", s, launch_ssd_decode(p, B, s));
    SSM_TIMED("m2.decode.group_sumsq", s, launch_ssd_group_sumsq(L.hs, (int)m.H, (int)(m.r * m.H), m.hpg, (int)m.G,
                                                                sumsq_partial, B, s));
    return SSM_OK;
}

int ssm2_shard_decode_stage2(const ssm2_shard_desc_t* d, const ssm2_shard_weights_t* w, const float* sumsq, int32_t B,
                             void* y, void* ws, size_t ws_bytes, hipStream_t s) {
    M2 m;
    SSM_TRY(m2_dims(d, &m));
    SSM_TRY(m2_check_weights(w));
    if (B < 0) return fail(SSM_E_INVAL, "batch %d", B);
    M2Ws L = m2_layout(m, B, 0, false, nullptr);
    SSM_TRY(check_ws(ws, ws_bytes, L.total));
    L = m2_layout(m, B, 0, false, ws);
    if (B == 0) return SSM_OK;
    SSM_TRY(check_ptr(sumsq, "sumsq"));
    SSM_TRY(check_ptr(y, "y_partial"));
    return m2_stage2(m, w, sumsq, B, y, L, s, "m2.decode.norm", "m2.decode.out_proj", "m2.decode.norm_out_proj");
}

}  // extern "C"

// ================================================================ layer around the mixer
namespace {

int check_dtype(int32_t t, const char* what) {
    if (t != SSM_F32 && t != SSM_BF16) return fail(SSM_E_INVAL, "%s dtype %d", what, t);
    return SSM_OK;
}

int check_norm_dim(int64_t d) {
    if (d <= 0 || d % 8 != 0 || d > residual_rmsnorm_max_dim())
        return fail(SSM_E_INVAL, "row width %lld: a multiple of 8 up to %d", (long long)d, residual_rmsnorm_max_dim());
    return SSM_OK;
}

int check_stack(const ssm_stack_desc_t* d, const ssm_shard_weights_t* layers, const float* const* norm_w,
                const float* final_w) {
    if (!d) return fail(SSM_E_INVAL, "stack desc is null");
    SSM_TRY(check_desc(&d->layer));
    if (d->layer.shard_count != 1)
        return fail(SSM_E_INVAL, "a stack runs at full width (shard_count 1); split layers go through the layer calls");
    if (d->n_layers < 1) return fail(SSM_E_INVAL, "n_layers %d", d->n_layers);
    if (!(d->norm_eps > 0.0f)) return fail(SSM_E_INVAL, "norm_eps must be positive");
    if (!(d->bcdt_eps >= 0.0f)) return fail(SSM_E_INVAL, "bcdt_eps must be >= 0");
    SSM_TRY(check_norm_dim(d->layer.d_model));
    if (!layers || !norm_w) return fail(SSM_E_INVAL, "layer arrays are null");
    for (int l = 0; l < d->n_layers; ++l) {
        SSM_TRY(check_weights(&layers[l]));
        SSM_TRY(check_ptr(norm_w[l], "norm_w[l]"));
    }
    return check_ptr(final_w, "final_norm_w");
}

// the stack's own buffers follow the layer's workspace
struct StackBufs {
    float* resid;   // [T][d_model] f32
    char* normed;   // [T][d_model] act
    char* y;        // [T][d_model] act
    size_t total;
};

StackBufs stack_bufs(const ssm_shard_desc_t* d, int64_t T, size_t layer_total, void* base) {
    StackBufs S{};
    char* b = (char*)base;
    size_t off = layer_total;
    auto take = [&](size_t bytes) { char* p = b ? b + off : nullptr; off += align256(bytes); return p; };
    S.resid = (float*)take((size_t)T * d->d_model * 4);
    S.normed = take((size_t)T * d->d_model * act_bytes(d));
    S.y = take((size_t)T * d->d_model * act_bytes(d));
    S.total = off;
    return S;
}

NormParts one_part(const void* p) {
    NormParts q{};
    q.p[0] = p;
    q.n = 1;
    return q;
}

}  // namespace

extern "C" {

int ssm_residual_rmsnorm(const void* base, int32_t base_dtype, const void* const* parts, int32_t n_parts,
                         int32_t parts_dtype, float* residual, const float* norm_w, float eps, void* normed,
                         int32_t normed_dtype, int64_t T, int32_t d, hipStream_t s) {
    SSM_TRY(check_dtype(base_dtype, "base"));
    SSM_TRY(check_dtype(parts_dtype, "parts"));
    SSM_TRY(check_dtype(normed_dtype, "normed"));
    SSM_TRY(check_norm_dim(d));
    if (T < 0 || T > INT32_MAX) return fail(SSM_E_INVAL, "rows %lld", (long long)T);
    if (n_parts < 0 || n_parts > kMaxNormParts) return fail(SSM_E_INVAL, "n_parts %d (0..%d)", n_parts, kMaxNormParts);
    if (!(eps > 0.0f)) return fail(SSM_E_INVAL, "eps must be positive");
    if (T == 0) return SSM_OK;
    SSM_TRY(check_ptr(base, "base"));
    SSM_TRY(check_ptr(residual, "residual"));
    SSM_TRY(check_ptr(norm_w, "norm_w"));
    SSM_TRY(check_ptr(normed, "normed"));
    NormParts q{};
    q.n = n_parts;
    if (n_parts > 0 && !parts) return fail(SSM_E_INVAL, "parts is null");
    for (int k = 0; k < n_parts; ++k) {
        SSM_TRY(check_ptr(parts[k], "parts[k]"));
        q.p[k] = parts[k];
    }
    if (base != residual && base_dtype == SSM_F32) {
        // distinct buffers must not overlap partially
        const char *b0 = (const char*)base, *r0 = (const char*)residual;
        const size_t n = (size_t)T * d * 4;
        if (b0 < r0 + n && r0 < b0 + n) return fail(SSM_E_INVAL, "base and residual overlap without being equal");
    }
    SSM_TIMED("layer.residual_rmsnorm", s,
              launch_residual_rmsnorm(base, base_dtype == SSM_BF16, q, parts_dtype == SSM_BF16, residual, norm_w, eps,
                                      normed, normed_dtype == SSM_BF16, T, d, s));
    return SSM_OK;
}

int ssm_bcdt_rmsnorm(float* x_dbl, int64_t T, int32_t R, int32_t N, int64_t ld, float eps, hipStream_t s) {
    if (T < 0 || R < 1 || N < 1 || ld < (int64_t)R + 2 * N) return fail(SSM_E_INVAL, "bcdt shape");
    if (!(eps > 0.0f)) return fail(SSM_E_INVAL, "eps must be positive");
    if (T == 0) return SSM_OK;
    if (!x_dbl) return fail(SSM_E_INVAL, "x_dbl is null");
    if (((uintptr_t)x_dbl & 3) != 0) return fail(SSM_E_ALIGN, "x_dbl is not 4-byte aligned");
    SSM_TIMED("layer.bcdt_rms", s, launch_bcdt_rms(x_dbl, T, R, N, ld, eps, s));
    return SSM_OK;
}

int ssm_stack_prefill_workspace_bytes(const ssm_stack_desc_t* desc, int64_t max_tokens, int32_t max_seqs,
                                      size_t* bytes) {
    if (!desc) return fail(SSM_E_INVAL, "stack desc is null");
    SSM_TRY(check_desc(&desc->layer));
    if (!bytes || max_tokens < 0 || max_tokens > INT32_MAX || max_seqs < 0) return fail(SSM_E_INVAL, "bad size query");
    const size_t lt = prefill_layout(&desc->layer, max_tokens, max_seqs, nullptr).total;
    *bytes = stack_bufs(&desc->layer, max_tokens, lt, nullptr).total;
    return SSM_OK;
}

int ssm_stack_decode_workspace_bytes(const ssm_stack_desc_t* desc, int32_t max_batch, size_t* bytes) {
    if (!desc) return fail(SSM_E_INVAL, "stack desc is null");
    SSM_TRY(check_desc(&desc->layer));
    if (!bytes || max_batch < 0) return fail(SSM_E_INVAL, "bad size query");
    const size_t lt = decode_layout(&desc->layer, max_batch, nullptr).total;
    *bytes = stack_bufs(&desc->layer, max_batch, lt, nullptr).total;
    return SSM_OK;
}

int ssm_stack_prefill(const ssm_stack_desc_t* sd, const ssm_shard_weights_t* layers, const float* const* norm_w,
                      const float* final_w, const void* x, int64_t T, const ssm_seq_meta_t* m,
                      void* const* conv_pools, float* const* ssm_pools, int32_t S, void* out, void* ws,
                      size_t ws_bytes, hipStream_t s) {
    SSM_TRY(check_stack(sd, layers, norm_w, final_w));
    const ssm_shard_desc_t* d = &sd->layer;
    PrefillWs L;
    SSM_TRY(prefill_checks(d, &layers[0], T, m, S, ws, ws_bytes, &L));
    const StackBufs B = stack_bufs(d, T, L.total, ws);
    SSM_TRY(check_ws(ws, ws_bytes, B.total));
    if (!conv_pools || !ssm_pools) return fail(SSM_E_INVAL, "pool arrays are null");
    for (int l = 0; l < sd->n_layers; ++l) {
        if (d->d_conv > 1) SSM_TRY(check_ptr(conv_pools[l], "conv_pools[l]"));
        SSM_TRY(check_ptr(ssm_pools[l], "ssm_pools[l]"));
    }
    if (T > 0) {
        SSM_TRY(check_ptr(x, "x"));
        SSM_TRY(check_ptr(out, "out"));
    }
    const bool bf = d->act_dtype == SSM_BF16;
    const int dm = d->d_model, R = d->dt_rank, N = d->d_state, W = R + 2 * N;
    const float eps = sd->norm_eps;
    NormParts none{};
    SSM_TIMED("layer.residual_rmsnorm", s,
              launch_residual_rmsnorm(x, bf, none, bf, B.resid, norm_w[0], eps, B.normed, bf, T, dm, s));
    for (int l = 0; l < sd->n_layers; ++l) {
        SSM_TRY(prefill1(d, &layers[l], B.normed, T, m, conv_pools[l], S, L.xdbl, L, s));
        if (sd->bcdt_eps > 0.0f) SSM_TIMED("layer.bcdt_rms", s, launch_bcdt_rms(L.xdbl, T, R, N, W, sd->bcdt_eps, s));
        SSM_TRY(prefill2(d, &layers[l], L.xdbl, T, m, ssm_pools[l], S, B.y, L, s));
        const bool last = l + 1 == sd->n_layers;
        SSM_TIMED("layer.residual_rmsnorm", s,
                  launch_residual_rmsnorm(B.resid, false, one_part(B.y), bf, B.resid, last ? final_w : norm_w[l + 1],
                                          eps, last ? out : B.normed, bf, T, dm, s));
    }
    return SSM_OK;
}

int ssm_stack_decode_step(const ssm_stack_desc_t* sd, const ssm_shard_weights_t* layers, const float* const* norm_w,
                          const float* final_w, const void* x, int32_t Bsz, const int32_t* slot,
                          void* const* conv_pools, float* const* ssm_pools, int32_t S, void* out, void* ws,
                          size_t ws_bytes, hipStream_t s) {
    SSM_TRY(check_stack(sd, layers, norm_w, final_w));
    const ssm_shard_desc_t* d = &sd->layer;
    DecodeWs L;
    SSM_TRY(decode_checks(d, &layers[0], Bsz, slot, S, ws, ws_bytes, &L));
    const StackBufs B = stack_bufs(d, Bsz, L.total, ws);
    SSM_TRY(check_ws(ws, ws_bytes, B.total));
    if (!conv_pools || !ssm_pools) return fail(SSM_E_INVAL, "pool arrays are null");
    for (int l = 0; l < sd->n_layers; ++l) {
        if (d->d_conv > 1) SSM_TRY(check_ptr(conv_pools[l], "conv_pools[l]"));
        SSM_TRY(check_ptr(ssm_pools[l], "ssm_pools[l]"));
    }
    if (Bsz == 0) return SSM_OK;
    SSM_TRY(check_ptr(x, "x_t"));
    SSM_TRY(check_ptr(out, "out"));
    const bool bf = d->act_dtype == SSM_BF16;
    const int dm = d->d_model, R = d->dt_rank, N = d->d_state, W = R + 2 * N;
    const float eps = sd->norm_eps;
    NormParts none{};
    SSM_TIMED("layer.residual_rmsnorm", s,
              launch_residual_rmsnorm(x, bf, none, bf, B.resid, norm_w[0], eps, B.normed, bf, Bsz, dm, s));
    for (int l = 0; l < sd->n_layers; ++l) {
        SSM_TRY(decode1(d, &layers[l], B.normed, Bsz, slot, conv_pools[l], S, L.xdbl, L, s));
        if (sd->bcdt_eps > 0.0f) SSM_TIMED("layer.bcdt_rms", s, launch_bcdt_rms(L.xdbl, Bsz, R, N, W, sd->bcdt_eps, s));
        SSM_TRY(decode2(d, &layers[l], L.xdbl, Bsz, slot, ssm_pools[l], S, B.y, L, s));
        const bool last = l + 1 == sd->n_layers;
        SSM_TIMED("layer.residual_rmsnorm", s,
                  launch_residual_rmsnorm(B.resid, false, one_part(B.y), bf, B.resid, last ? final_w : norm_w[l + 1],
                                          eps, last ? out : B.normed, bf, Bsz, dm, s));
    }
    return SSM_OK;
}

}  // extern "C"
