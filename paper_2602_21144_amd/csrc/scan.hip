// Selective scan of the SSM path (Section II-B; Section IV-C: Delta sharded with the
// channels, B and C complete on every rank, A and D local) and the recurrent half of
// the SSM cache (Section IV-A).
//
// Per channel c and state n:  Delta_t = softplus(dt_t + b_dt)
//                             h_t = exp(Delta_t * A) * h_{t-1} + Delta_t * B_t * u_t
//                             y_t = sum_n C_t[n] h_t[n] + D u_t ;  g_t = y_t * SiLU(z_t)
//
// Layout on gfx950: one lane per channel, its 16 fp32 states in VGPRs; B_t and C_t are
// the same for every channel of a token, so a workgroup stages them once per block of
// tokens in LDS and every lane reads them as broadcasts. The
// packed token range is cut into windows of `win` tokens so that there are enough
// waves for the 1024 SIMDs: pass A computes, for each window whose last sequence runs
// on into the next window, that piece's end state from a zero start (and its sum of
// Delta); pass B links windows in order per (channel, state) -- the state entering
// window j+1 is exp(A * sum Delta_j) * (state entering j) + local end state of j; pass C
// runs the full recurrence from the linked state and writes g and the final states.
// Pass A also stores Delta of every token of its window (it needs Delta for most of
// them anyway), so pass C reads it and runs no softplus.
// Initial states of continuing sequences are copied out of the pool in pass A, so pass
// C (which writes final states into the pool) never reads a slot another pass writes.
#include "common.h"

namespace ssm {
namespace {

constexpr int kWave = 64;
constexpr int kMinWin = 32, kMaxWin = 2048;
constexpr int kTargetWaves = 3072;  // 3 per SIMD: the main pass holds 156 VGPRs per lane

// flags per window, written by pass A
constexpr int kFlagContIn = 1;    // first token continues a sequence begun earlier
constexpr int kFlagCarryOut = 2;  // last sequence continues past the window end
constexpr int kFlagLastCont = 4;  // last piece starts at the window start as a continuation

__device__ __forceinline__ int uni(int v) { return __builtin_amdgcn_readfirstlane(v); }

__device__ __forceinline__ int seq_of(const int32_t* cu, int nseq, int64_t t) {
    int lo = 0, hi = nseq;
    while (hi - lo > 1) {
        int mid = (lo + hi) >> 1;
        if (cu[mid] <= t) lo = mid; else hi = mid;
    }
    return lo;
}

int64_t target_windows(int E) { return std::max<int64_t>(1, (int64_t)kTargetWaves * kWave / E); }

constexpr int kTB = 8;  // tokens per block: loads for block i+1 are in flight while block i computes

// Per-lane activations of one block of tokens, prefetched a block ahead: u and dt for
// pass A; u, the stored Delta and z for pass C.
template <typename T, bool MAIN>
struct TokBlock {
    T u[kTB], dt[MAIN ? 1 : kTB], z[MAIN ? kTB : 1];
    float delta[MAIN ? kTB : 1];
    __device__ __forceinline__ void load(const ScanArgs& a, int64_t b0, int64_t w1, int c) {
#pragma unroll
        for (int i = 0; i < kTB; ++i) {
            const int64_t t = b0 + i < w1 ? b0 + i : w1 - 1;  // clamp: tail entries are never used
            u[i] = ((const T*)a.u)[t * a.E + c];
            if constexpr (MAIN) {
                delta[i] = a.delta[t * a.E + c];
                z[i] = ((const T*)a.z)[t * a.ld_z + c];
            } else {
                dt[i] = ((const T*)a.dt)[t * a.E + c];
            }
        }
    }
};

// B_t and C_t of a block of tokens (2N floats each), staged once per workgroup in LDS.
// Threads 0..kTB*8-1 each move one float4; all lanes then read them as broadcasts.
struct BcStage {
    float4 v;
    __device__ __forceinline__ void load(const ScanArgs& a, int64_t b0, int64_t w1, int tid, int nthreads) {
        if (tid < kTB * 8) {
            const int i = tid >> 3, q = tid & 7;
            const int64_t t = b0 + i < w1 ? b0 + i : w1 - 1;
            v = *(const float4*)(a.xdbl + t * a.ld_xdbl + a.R + 4 * q);
        }
        (void)nthreads;
    }
    __device__ __forceinline__ void store(float (*lds)[2 * kN], int tid) const {
        if (tid < kTB * 8) *(float4*)&lds[tid >> 3][4 * (tid & 7)] = v;
    }
};

__device__ __forceinline__ void load_h(float* h, const float* src) {
#pragma unroll
    for (int q = 0; q < kN / 4; ++q) {
        const float4 v = ((const float4*)src)[q];
        h[4 * q] = v.x; h[4 * q + 1] = v.y; h[4 * q + 2] = v.z; h[4 * q + 3] = v.w;
    }
}
__device__ __forceinline__ void store_h(float* dst, const float* h) {
#pragma unroll
    for (int q = 0; q < kN / 4; ++q) ((float4*)dst)[q] = make_float4(h[4 * q], h[4 * q + 1], h[4 * q + 2], h[4 * q + 3]);
}

// ---------------------------------------------------------------- pass A
template <typename T, int CW>
__global__ __launch_bounds__(kWave * CW) void scan_local_kernel(ScanArgs a, int nwin, int32_t* wflags) {
    __shared__ float bc[2][kTB][2 * kN];
    const int cblocks = a.E / (kWave * CW);
    const int j = blockIdx.x / cblocks;
    const int tid = threadIdx.x;
    const int c = (blockIdx.x % cblocks) * kWave * CW + tid;
    const int64_t w0 = (int64_t)j * a.win, w1 = min(w0 + a.win, a.T);
    const int s_first = uni(seq_of(a.cu, a.nseq, w0));
    const int s_last = uni(seq_of(a.cu, a.nseq, w1 - 1));
    const int64_t b_first = uni(a.cu[s_first]);
    const int64_t b_last = uni(a.cu[s_last]), e_last = uni(a.cu[s_last + 1]);
    const bool carry_out = w1 < a.T && e_last > w1;
    const bool last_cont = b_last < w0;
    if (blockIdx.x % cblocks == 0 && tid == 0)
        wflags[j] = (b_first < w0 ? kFlagContIn : 0) | (carry_out ? kFlagCarryOut : 0) | (last_cont ? kFlagLastCont : 0);

    // copy the initial state of every non-empty sequence that starts in this window
    for (int s = s_first; s <= s_last; ++s) {
        const int64_t b = uni(a.cu[s]), e = uni(a.cu[s + 1]);
        if (b < w0 || e <= b || !a.has_init[s]) continue;
        const int slot = uni(a.slot[s]);
        if (slot < 0 || slot >= a.S) {
            if (tid == 0) atomicOr(a.status, SSM_STATUS_BAD_SLOT);
            continue;
        }
        float h[kN];
        load_h(h, a.pool + ((int64_t)slot * a.E + c) * kN);
        store_h(a.h0_seq + ((int64_t)s * a.E + c) * kN, h);
    }

    // Delta of the tokens before the piece whose recurrence runs here (all of them when
    // no piece carries out of the window)
    const float bdt = a.b_dt[c];
    const int64_t t0 = !carry_out ? w1 : last_cont ? w0 : b_last;
    for (int64_t b0 = w0; b0 < t0; b0 += kTB) {
        T dtv[kTB];
#pragma unroll
        for (int i = 0; i < kTB; ++i) {
            const int64_t t = b0 + i < t0 ? b0 + i : t0 - 1;
            dtv[i] = ((const T*)a.dt)[t * a.E + c];
        }
#pragma unroll
        for (int i = 0; i < kTB; ++i)
            if (b0 + i < t0) a.delta[(b0 + i) * a.E + c] = softplus_f(to_f32(dtv[i]) + bdt);
    }
    if (!carry_out) return;

    // local end state of the last piece: from zero if it continues an earlier window,
    // else from the sequence's own initial state
    float A2[kN], h[kN];
#pragma unroll
    for (int n = 0; n < kN; ++n) A2[n] = -__expf(a.A_log[c * kN + n]) * kLog2e;
    if (!last_cont && a.has_init[s_last]) {
        const int slot = uni(a.slot[s_last]);
        if (slot >= 0 && slot < a.S) load_h(h, a.pool + ((int64_t)slot * a.E + c) * kN);
        else
#pragma unroll
            for (int n = 0; n < kN; ++n) h[n] = 0.0f;
    } else {
#pragma unroll
        for (int n = 0; n < kN; ++n) h[n] = 0.0f;
    }
    float sum_delta = 0.0f;
    TokBlock<T, false> nxt;
    BcStage st;
    nxt.load(a, t0, w1, c);
    st.load(a, t0, w1, tid, kWave * CW);
    st.store(bc[0], tid);
    __syncthreads();
    int buf = 0;
    for (int64_t b0 = t0; b0 < w1; b0 += kTB) {
        const TokBlock<T, false> cur = nxt;
        const bool more = b0 + kTB < w1;
        if (more) {
            nxt.load(a, b0 + kTB, w1, c);
            st.load(a, b0 + kTB, w1, tid, kWave * CW);
        }
        const int nt = rows_upto(w1 - b0, kTB);
        auto step = [&](int i) {
            const float delta = softplus_f(to_f32(cur.dt[i]) + bdt);
            a.delta[(b0 + i) * a.E + c] = delta;
            const float du = delta * to_f32(cur.u[i]);
            sum_delta += delta;
#pragma unroll
            for (int n = 0; n < kN; ++n) h[n] = fast_exp2(delta * A2[n]) * h[n] + du * bc[buf][i][n];
        };
        if (nt == kTB) {
#pragma unroll
            for (int i = 0; i < kTB; ++i) step(i);
        } else {
#pragma unroll
            for (int i = 0; i < kTB; ++i)
                if (i < nt) step(i);
        }
        if (more) st.store(bc[buf ^ 1], tid);
        __syncthreads();
        buf ^= 1;
    }
    store_h(a.h_local + ((int64_t)j * a.E + c) * kN, h);
    a.sum_delta[(int64_t)j * a.E + c] = sum_delta;
}

// ---------------------------------------------------------------- pass B
// Window j maps the state carried across its start to the one carried across its end by
// x -> m x + l: (exp(A * sum Delta_j), local end state) when its last piece continues from
// its start, (0, local end state) when that piece starts inside it, (1, 0) when nothing
// carries out. The windows of a (channel, state) are cut into kLinkSeg ranges, one lane
// each: a lane composes its range's maps, takes its entry state from the composites of
// the ranges before it (through LDS), then walks its range again from that entry, writing
// the linked entry state of every window whose first token continues a sequence. The
// serial chain is thus one range long instead of all windows. Also clears the state of
// empty sequences that start fresh (their final state is the zero initial state).
constexpr int kLinkSeg = 8;     // ranges per (channel, state): one wave each
constexpr int kLinkPairs = 64;  // (channel, state) pairs per workgroup: one per lane
constexpr int kLB = 8;          // windows fetched at a time, so that only the chain itself is serial

__global__ __launch_bounds__(kLinkSeg * kLinkPairs) void scan_link_kernel(ScanArgs a, int nwin,
                                                                          const int32_t* wflags) {
    __shared__ float cm[kLinkSeg][kLinkPairs], cl[kLinkSeg][kLinkPairs];
    const int p = threadIdx.x % kLinkPairs, r = uni(threadIdx.x / kLinkPairs);
    const int64_t pair = (int64_t)blockIdx.x * kLinkPairs + p;
    const bool live = pair < (int64_t)a.E * kN;
    const int c = live ? (int)(pair / kN) : 0, n = live ? (int)(pair % kN) : 0;
    const float A2 = -__expf(a.A_log[c * kN + n]) * kLog2e;
    const int per = (nwin + kLinkSeg - 1) / kLinkSeg;
    const int j_beg = min(r * per, nwin), j_end = min(j_beg + per, nwin);

    // one batch of the range's windows: flags, decay exp(A * sum Delta) and local end
    // state (entries of windows without a carry are never written by pass A and are read
    // but not used)
    int fl[kLB];
    float dd[kLB], hl[kLB];
    auto fetch = [&](int j0) {
#pragma unroll
        for (int q = 0; q < kLB; ++q) {
            if (j0 + q >= j_end) break;
            const int64_t j = j0 + q;
            fl[q] = wflags[j];
            hl[q] = a.h_local[(j * a.E + c) * kN + n];
            dd[q] = a.sum_delta[j * a.E + c];
        }
#pragma unroll
        for (int q = 0; q < kLB; ++q) {
            if (j0 + q >= j_end) break;
            dd[q] = fast_exp2(dd[q] * A2);
        }
    };

    // this range's composite map
    float m = 1.0f, l = 0.0f;
    for (int j0 = j_beg; j0 < j_end; j0 += kLB) {
        fetch(j0);
#pragma unroll
        for (int q = 0; q < kLB; ++q) {
            if (j0 + q >= j_end) break;
            if (fl[q] & kFlagCarryOut) {
                if (fl[q] & kFlagLastCont) { m *= dd[q]; l = dd[q] * l + hl[q]; }
                else { m = 0.0f; l = hl[q]; }
            }
        }
    }
    cm[r][p] = m;
    cl[r][p] = l;
    __syncthreads();
    float carry = 0.0f;
    for (int q = 0; q < r; ++q) carry = cm[q][p] * carry + cl[q][p];

    // walk the range again from its entry (a range of one batch still holds it)
    const bool refetch = j_end - j_beg > kLB;
    for (int j0 = j_beg; j0 < j_end; j0 += kLB) {
        if (refetch) fetch(j0);
#pragma unroll
        for (int q = 0; q < kLB; ++q) {
            if (j0 + q >= j_end) break;
            if ((fl[q] & kFlagContIn) && live) a.h_in[((int64_t)(j0 + q) * a.E + c) * kN + n] = carry;
            if (fl[q] & kFlagCarryOut) carry = (fl[q] & kFlagLastCont) ? dd[q] * carry + hl[q] : hl[q];
        }
    }

    if (!live) return;
    for (int s = r; s < a.nseq; s += kLinkSeg) {  // the ranges' waves share the sequences
        if (a.cu[s + 1] != a.cu[s] || a.has_init[s]) continue;
        const int slot = a.slot[s];
        if (slot < 0 || slot >= a.S) continue;
        a.pool[((int64_t)slot * a.E + c) * kN + n] = 0.0f;
    }
}

// ---------------------------------------------------------------- pass C
// One token of the full recurrence for this lane's channel; returns g.
__device__ __forceinline__ float token_step(float* h, const float* A2, float u, float delta, float z, float Dc,
                                            const float* bcrow) {
    const float du = delta * u;
    float y = 0.0f;
#pragma unroll
    for (int n = 0; n < kN; ++n) {
        h[n] = fast_exp2(delta * A2[n]) * h[n] + du * bcrow[n];
        y += bcrow[kN + n] * h[n];
    }
    y += Dc * u;
    return y * silu_f(z);
}

template <typename T, int CW>
__global__ __launch_bounds__(kWave * CW) void scan_main_kernel(ScanArgs a) {
    __shared__ float bc[2][kTB][2 * kN];
    const int cblocks = a.E / (kWave * CW);
    const int j = blockIdx.x / cblocks;
    const int tid = threadIdx.x;
    const int c = (blockIdx.x % cblocks) * kWave * CW + tid;
    const int64_t w0 = (int64_t)j * a.win, w1 = min(w0 + a.win, a.T);
    float A2[kN], h[kN];
#pragma unroll
    for (int n = 0; n < kN; ++n) A2[n] = -__expf(a.A_log[c * kN + n]) * kLog2e;
    const float Dc = a.D[c];
    T* g = (T*)a.g;

    // the sequence holding the first token, and the state entering the window
    int s = uni(seq_of(a.cu, a.nseq, w0));
    int64_t s_beg = uni(a.cu[s]), s_end = uni(a.cu[s + 1]);
    if (s_beg < w0) {
        load_h(h, a.h_in + ((int64_t)j * a.E + c) * kN);
    } else if (a.has_init[s]) {
        load_h(h, a.h0_seq + ((int64_t)s * a.E + c) * kN);
    } else {
#pragma unroll
        for (int n = 0; n < kN; ++n) h[n] = 0.0f;
    }
    bool ok = true;  // false once cu_seqlens proves inconsistent

    TokBlock<T, true> nxt;
    BcStage st;
    nxt.load(a, w0, w1, c);
    st.load(a, w0, w1, tid, kWave * CW);
    st.store(bc[0], tid);
    __syncthreads();
    int buf = 0;
    for (int64_t b0 = w0; b0 < w1; b0 += kTB) {
        const TokBlock<T, true> cur = nxt;
        const bool more = b0 + kTB < w1;
        if (more) {
            nxt.load(a, b0 + kTB, w1, c);
            st.load(a, b0 + kTB, w1, tid, kWave * CW);
        }
        const int nt = rows_upto(w1 - b0, kTB);
        if (ok && s_end >= b0 + nt) {
            // no sequence ends inside this block: straight-line recurrence from registers
            // (a whole block without per-token guards, so the states stay in place)
            auto step = [&](int i) {
                g[(b0 + i) * a.E + c] = from_f32<T>(token_step(h, A2, to_f32(cur.u[i]), cur.delta[i],
                                                               to_f32(cur.z[i]), Dc, bc[buf][i]));
            };
            if (nt == kTB) {
#pragma unroll
                for (int i = 0; i < kTB; ++i) step(i);
            } else {
#pragma unroll
                for (int i = 0; i < kTB; ++i)
                    if (i < nt) step(i);
            }
        } else if (ok) {
            // a sequence ends in this block: store its state, start the next one (empty
            // sequences are left to the link pass); operands are re-read by token index
#pragma unroll 1
            for (int i = 0; i < nt && ok; ++i) {
                const int64_t t = b0 + i;
                while (t >= s_end) {
                    if (s_end < t || s + 1 >= a.nseq) {
                        ok = false;
                        if (tid == 0) atomicOr(a.status, SSM_STATUS_BAD_SEQLENS);
                        break;
                    }
                    if (s_end > s_beg) {
                        const int slot = uni(a.slot[s]);
                        if (slot >= 0 && slot < a.S) store_h(a.pool + ((int64_t)slot * a.E + c) * kN, h);
                        else if (tid == 0) atomicOr(a.status, SSM_STATUS_BAD_SLOT);
                    }
                    ++s;
                    s_beg = uni(a.cu[s]);
                    s_end = uni(a.cu[s + 1]);
                    if (s_end > s_beg && a.has_init[s]) {
                        load_h(h, a.h0_seq + ((int64_t)s * a.E + c) * kN);
                    } else {
#pragma unroll
                        for (int n = 0; n < kN; ++n) h[n] = 0.0f;
                    }
                }
                if (!ok) break;
                const float u = to_f32(((const T*)a.u)[t * a.E + c]);
                const float delta = a.delta[t * a.E + c];
                const float z = to_f32(((const T*)a.z)[t * a.ld_z + c]);
                g[t * a.E + c] = from_f32<T>(token_step(h, A2, u, delta, z, Dc, bc[buf][i]));
            }
        }
        if (more) st.store(bc[buf ^ 1], tid);
        __syncthreads();
        buf ^= 1;
    }
    // a sequence ending exactly at the window end stores its state here
    if (ok && s_end == w1 && s_end > s_beg) {
        const int slot = uni(a.slot[s]);
        if (slot >= 0 && slot < a.S) store_h(a.pool + ((int64_t)slot * a.E + c) * kN, h);
        else if (tid == 0) atomicOr(a.status, SSM_STATUS_BAD_SLOT);
    }
}

// ---------------------------------------------------------------- decode
// One recurrence step on the cached states, in place. Four lanes share a (sequence,
// channel): lane q holds states 4q..4q+3 as one float4, so a wave reads and writes 16
// channels x 64 bytes = 1 KB contiguous per instruction (a lane per channel would touch
// 16 bytes of every 64 across 4 KB). The channel's y is summed over the four lanes by
// two xor shuffles; the first lane of each group applies the D skip and the gate.
template <typename T>
__global__ __launch_bounds__(256) void decode_ssm_kernel(ScanArgs a) {
    const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t item = gid >> 2;  // (sequence, channel)
    const int q = (int)(gid & 3);
    // every lane of a quad takes part in the shuffles: items past the end compute on a
    // clamped item and store nothing
    const bool live = item < (int64_t)a.nseq * a.E;
    const int64_t itc = live ? item : 0;
    const int b = (int)(itc / a.E), c = (int)(itc % a.E);
    const int slot = a.slot[b];
    // everything that does not depend on the slot goes out with the slot index, before the
    // slot-addressed state
    const float4 al = ((const float4*)(a.A_log + (int64_t)c * kN))[q];
    const float* xb = a.xdbl + (int64_t)b * a.ld_xdbl + a.R;  // B at 0, C at kN (16-byte aligned)
    const float4 Bq = ((const float4*)xb)[q], Cq = ((const float4*)(xb + kN))[q];
    const float u = to_f32(((const T*)a.u)[(int64_t)b * a.E + c]);
    const float dt = to_f32(((const T*)a.dt)[(int64_t)b * a.E + c]);
    const float z = to_f32(((const T*)a.z)[(int64_t)b * a.ld_z + c]);
    const float bdt = a.b_dt[c], Dc = a.D[c];
    __builtin_amdgcn_sched_barrier(0);
    const bool slot_ok = slot >= 0 && slot < a.S;
    float4* hp = (float4*)(a.pool + ((int64_t)(slot_ok ? slot : 0) * a.E + c) * kN) + q;
    const float4 h = *hp;
    const float delta = softplus_f(dt + bdt);
    const float du = delta * u;
    const float hv[4] = {h.x, h.y, h.z, h.w}, av[4] = {al.x, al.y, al.z, al.w};
    const float bv[4] = {Bq.x, Bq.y, Bq.z, Bq.w}, cv[4] = {Cq.x, Cq.y, Cq.z, Cq.w};
    float hn[4], y = 0.0f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        hn[i] = fast_exp2(delta * (-__expf(av[i]) * kLog2e)) * hv[i] + du * bv[i];
        y += cv[i] * hn[i];
    }
    y += __shfl_xor(y, 1);
    y += __shfl_xor(y, 2);
    // z and D are used only past the exits below; keeping them live here stops the compiler
    // from sinking their loads behind the exits (a second memory round trip per wave)
    asm volatile("" ::"v"(z), "v"(Dc));
    if (!live) return;
    if (!slot_ok) {
        if (q == 0) {
            atomicOr(a.status, SSM_STATUS_BAD_SLOT);
            ((T*)a.g)[(int64_t)b * a.E + c] = from_f32<T>(0.0f);
        }
        return;
    }
    *hp = make_float4(hn[0], hn[1], hn[2], hn[3]);
    if (q == 0) ((T*)a.g)[(int64_t)b * a.E + c] = from_f32<T>((y + Dc * u) * silu_f(z));
}

// The large-batch state step with dt_proj fused in: four lanes per (sequence, channel)
// first form dt = sum_r delta[r] * W_dt[c][r] (delta rounded to the activation dtype, as
// dt_proj's operand; lane q takes the 8-wide chunks q, q + 4, ... of the R columns, the
// quad sums them with two shuffles), round dt to the activation dtype as dt_proj stores
// it, then take the step of decode_ssm_kernel. One launch and no dt round trip instead of
// a dt_proj GEMM followed by the state kernel.
// A workgroup takes 16 channels of 4 sequences (64 items, four lanes each): each W_dt row
// serves the 4 sequences of one workgroup instead of being fetched per sequence, and each
// wave's states are one sequence's 16 channels, 1 KB contiguous per load instruction (with
// 8 x 8 tiles, two 512-byte runs per instruction, the step took 15.7 instead of 10 us).
constexpr int kDtCh = 16, kDtSeq = 4;  // tiles of the fp32 / general state-step kernel
constexpr int kDtSeqM = 16;            // sequences per tile of the bf16 MFMA state-step kernel
constexpr int kDtSpw = 2;              // sequences per wave of that kernel

// bf16 and dt_rank a multiple of 32 (up to 512): a workgroup takes CT tiles of 16 channels
// (adjacent, so they share the delta rows and B, C) of 16 sequences, SPW sequences per wave
// (four lanes per (sequence, channel), a float4 of states each: every state load and store
// instruction covers 1 KB contiguous). The step is bound by the state bytes in flight over the
// memory latency; for 256 sequences of 1280 channels one sequence per wave took 13.1 us, two
// 12.5 us, four 14.3 us; two tiles per workgroup (640 workgroups, one round at 76 VGPRs and
// three workgroups per CU, instead of 1280 in 1.25 rounds) 11.7 us. Each tile's 16 x 16 dt is
// the product delta[16 sequences][R] x W_dt[16 channels][R]^T: k-chunk k of the R / 32 is one
// v_mfma_f32_16x16x32_bf16 on wave k % (waves); the waves' partial tiles meet in LDS, every
// thread adds them in wave order and rounds dt to bf16 as dt_proj stores it. Each workgroup
// fetches its 16 delta rows and its W_dt rows once. (4 x 16 tiles fetched the W_dt rows once
// per 4 sequences, about as many L2 bytes as the states themselves: 15.5 us.)
template <int NK, int SPW, int CT>
__global__ __launch_bounds__(64 * kDtSeqM / SPW) void decode_dt_ssm_mfma_kernel(ScanArgs a) {
    constexpr int NWV = kDtSeqM / SPW;         // waves
    constexpr int KPW = (NK + NWV - 1) / NWV;  // k-chunks per wave
    constexpr int NP = NK < NWV ? NK : NWV;    // partial tiles
    __shared__ float dt_part[CT][NP][kDtSeqM][kDtCh];
    const int cgroups = a.E / (kDtCh * CT);
    const int tb = blockIdx.x / cgroups, tg = blockIdx.x % cgroups;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int it = lane >> 2, q = lane & 3;  // channel (tg CT + t) 16 + it of tile t; states 4q .. 4q + 3
    int bsq[SPW], slot[SPW];
    bool live[SPW], sok[SPW];
    float4 Bq[SPW], Cq[SPW], h[CT][SPW];
    float u[CT][SPW], z[CT][SPW];
    // the slot indices first: the state loads wait for them alone
#pragma unroll
    for (int j = 0; j < SPW; ++j) {
        const int bb = tb * kDtSeqM + SPW * wave + j;
        live[j] = bb < a.nseq;
        bsq[j] = live[j] ? bb : 0;
        slot[j] = a.slot[bsq[j]];
    }
    // the dt tiles' operands, issued before the states so that the MFMAs wait for them and
    // not for the states (which stay in flight across the dt tiles and the barrier). Chunks
    // k = wave + NWV kk: lane l takes delta row l % 16 (rows past the batch zero; shared by
    // the CT tiles) and W_dt row l % 16 of each tile, columns 32 k + 8 (l / 16) .. + 7
    const bool mw = wave < NK;
    const int r = lane & 15, kq = (lane >> 4) * 8;
    const bool rok = tb * kDtSeqM + r < a.nseq;
    // every wave issues them (waves past the last chunk re-read chunk 0, unused), so that no
    // branch hides the loads' count from the compiler's counter waits
    float4 d0[KPW], d1[KPW];
    bf16x8 wf[CT][KPW];
    {
        const float* drow = a.xdbl + (int64_t)(rok ? tb * kDtSeqM + r : 0) * a.ld_xdbl;
#pragma unroll
        for (int kk = 0; kk < KPW; ++kk) {
            const int k = wave + NWV * kk < NK ? wave + NWV * kk : 0;  // past the last chunk: re-read, not added
            d0[kk] = *(const float4*)(drow + 32 * k + kq);
            d1[kk] = *(const float4*)(drow + 32 * k + kq + 4);
#pragma unroll
            for (int t = 0; t < CT; ++t)
                wf[t][kk] = *(const bf16x8*)((const bf16*)a.w_dt + (int64_t)((tg * CT + t) * kDtCh + r) * a.R + 32 * k + kq);
        }
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int j = 0; j < SPW; ++j) {
        sok[j] = slot[j] >= 0 && slot[j] < a.S;
#pragma unroll
        for (int t = 0; t < CT; ++t)
            h[t][j] = ((const float4*)(a.pool + ((int64_t)(sok[j] ? slot[j] : 0) * a.E + (tg * CT + t) * kDtCh + it) * kN))[q];
    }
    __builtin_amdgcn_sched_barrier(0);
    if (mw) {
#pragma unroll
        for (int t = 0; t < CT; ++t) {
            f32x4 acc = f32x4{};
#pragma unroll
            for (int kk = 0; kk < KPW; ++kk) {
                bf16x8 af;
                af[0] = (bf16)d0[kk].x; af[1] = (bf16)d0[kk].y; af[2] = (bf16)d0[kk].z; af[3] = (bf16)d0[kk].w;
                af[4] = (bf16)d1[kk].x; af[5] = (bf16)d1[kk].y; af[6] = (bf16)d1[kk].z; af[7] = (bf16)d1[kk].w;
                if (!rok || wave + NWV * kk >= NK) af = bf16x8{};
                acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af, wf[t][kk], acc, 0, 0, 0);
            }
            // lane l holds sequences 4 (l / 16) + j of the tile, channel l % 16
#pragma unroll
            for (int j = 0; j < 4; ++j) dt_part[t][wave][4 * (lane >> 4) + j][r] = acc[j];
        }
    }
    // the operands of the output alone, in flight across the barrier
#pragma unroll
    for (int j = 0; j < SPW; ++j) {
        const float* xb = a.xdbl + (int64_t)bsq[j] * a.ld_xdbl + a.R;
        Bq[j] = ((const float4*)xb)[q];
        Cq[j] = ((const float4*)(xb + kN))[q];
#pragma unroll
        for (int t = 0; t < CT; ++t) {
            const int c = (tg * CT + t) * kDtCh + it;
            u[t][j] = (float)((const bf16*)a.u)[(int64_t)bsq[j] * a.E + c];
            z[t][j] = (float)((const bf16*)a.z)[(int64_t)bsq[j] * a.ld_z + c];
        }
    }
    __syncthreads();
#pragma unroll
    for (int t = 0; t < CT; ++t) {
        const int c = (tg * CT + t) * kDtCh + it;
        const float4 al = ((const float4*)(a.A_log + (int64_t)c * kN))[q];
        const float bdt = a.b_dt[c], Dc = a.D[c];
        const float av[4] = {al.x, al.y, al.z, al.w};
#pragma unroll
        for (int j = 0; j < SPW; ++j) {
            const int ts = SPW * wave + j;
            float dsum = dt_part[t][0][ts][it];
#pragma unroll
            for (int k = 1; k < NP; ++k) dsum += dt_part[t][k][ts][it];
            const float dt = (float)(bf16)dsum;  // stored in bf16 as dt_proj's output
            const float delta = softplus_f(dt + bdt);
            const float du = delta * u[t][j];
            const float hv[4] = {h[t][j].x, h[t][j].y, h[t][j].z, h[t][j].w};
            const float bv[4] = {Bq[j].x, Bq[j].y, Bq[j].z, Bq[j].w}, cv[4] = {Cq[j].x, Cq[j].y, Cq[j].z, Cq[j].w};
            float hn[4], y = 0.0f;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                hn[i] = fast_exp2(delta * (-__expf(av[i]) * kLog2e)) * hv[i] + du * bv[i];
                y += cv[i] * hn[i];
            }
            y += __shfl_xor(y, 1);
            y += __shfl_xor(y, 2);
            if (!live[j]) continue;
            if (!sok[j]) {
                if (q == 0) {
                    atomicOr(a.status, SSM_STATUS_BAD_SLOT);
                    ((bf16*)a.g)[(int64_t)bsq[j] * a.E + c] = (bf16)0.0f;
                }
                continue;
            }
            ((float4*)(a.pool + ((int64_t)slot[j] * a.E + c) * kN))[q] = make_float4(hn[0], hn[1], hn[2], hn[3]);
            if (q == 0) ((bf16*)a.g)[(int64_t)bsq[j] * a.E + c] = (bf16)((y + Dc * u[t][j]) * silu_f(z[t][j]));
        }
    }
}

template <typename T, int NCH>
__global__ __launch_bounds__(256) void decode_dt_ssm_kernel(ScanArgs a) {
    const int ctiles = a.E / kDtCh;
    const int tb = blockIdx.x / ctiles, tc = blockIdx.x % ctiles;
    const int it = threadIdx.x >> 2, q = threadIdx.x & 3;
    const int bb = tb * kDtSeq + it / kDtCh, cc = tc * kDtCh + it % kDtCh;
    const bool live = bb < a.nseq;
    const int b = live ? bb : 0, c = cc;
    const int slot = a.slot[b];
    const float4 al = ((const float4*)(a.A_log + (int64_t)c * kN))[q];
    const float* xrow = a.xdbl + (int64_t)b * a.ld_xdbl;
    const float* xb = xrow + a.R;  // B at 0, C at kN (16-byte aligned)
    const float4 Bq = ((const float4*)xb)[q], Cq = ((const float4*)(xb + kN))[q];
    const float u = to_f32(((const T*)a.u)[(int64_t)b * a.E + c]);
    const float z = to_f32(((const T*)a.z)[(int64_t)b * a.ld_z + c]);
    const float bdt = a.b_dt[c], Dc = a.D[c];
    // dt operands: 8-column chunks q, q + 4, ... (at most NCH per lane), all issued at once;
    // chunks past R / 8 re-read chunk q and are not added
    const int nch = a.R / 8;
    const T* wrow = (const T*)a.w_dt + (int64_t)c * a.R;
    float4 d0[NCH], d1[NCH];
    u32x4 w0[NCH], w1[NCH];  // raw weights: 8 bf16 in w0, or 8 floats in w0 and w1
#pragma unroll
    for (int k = 0; k < NCH; ++k) {
        const int j = q + 4 * k < nch ? q + 4 * k : q;
        d0[k] = *(const float4*)(xrow + 8 * j);
        d1[k] = *(const float4*)(xrow + 8 * j + 4);
        w0[k] = *(const u32x4*)(wrow + 8 * j);
        if constexpr (sizeof(T) == 4) w1[k] = *(const u32x4*)(wrow + 8 * j + 4);
    }
    // the slot-addressed state goes out with the rest, before any of it is used
    const bool slot_ok = slot >= 0 && slot < a.S;
    float4* hp = (float4*)(a.pool + ((int64_t)(slot_ok ? slot : 0) * a.E + c) * kN) + q;
    const float4 h = *hp;
    __builtin_amdgcn_sched_barrier(0);
    float dt = 0.0f;
#pragma unroll
    for (int k = 0; k < NCH; ++k) {
        if (q + 4 * k < nch) {
            const float dv[8] = {d0[k].x, d0[k].y, d0[k].z, d0[k].w, d1[k].x, d1[k].y, d1[k].z, d1[k].w};
            float wv[8];
            if constexpr (sizeof(T) == 2) {
                const bf16x8 w8 = __builtin_bit_cast(bf16x8, w0[k]);
#pragma unroll
                for (int e = 0; e < 8; ++e) wv[e] = (float)w8[e];
            } else {
                const f32x4 a0 = __builtin_bit_cast(f32x4, w0[k]), a1 = __builtin_bit_cast(f32x4, w1[k]);
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    wv[e] = a0[e];
                    wv[4 + e] = a1[e];
                }
            }
#pragma unroll
            for (int e = 0; e < 8; ++e) dt += to_f32(from_f32<T>(dv[e])) * wv[e];
        }
    }
    dt += __shfl_xor(dt, 1);
    dt += __shfl_xor(dt, 2);
    dt = to_f32(from_f32<T>(dt));
    const float delta = softplus_f(dt + bdt);
    const float du = delta * u;
    const float hv[4] = {h.x, h.y, h.z, h.w}, av[4] = {al.x, al.y, al.z, al.w};
    const float bv[4] = {Bq.x, Bq.y, Bq.z, Bq.w}, cv[4] = {Cq.x, Cq.y, Cq.z, Cq.w};
    float hn[4], y = 0.0f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        hn[i] = fast_exp2(delta * (-__expf(av[i]) * kLog2e)) * hv[i] + du * bv[i];
        y += cv[i] * hn[i];
    }
    y += __shfl_xor(y, 1);
    y += __shfl_xor(y, 2);
    asm volatile("" ::"v"(z), "v"(Dc));
    if (!live) return;
    if (!slot_ok) {
        if (q == 0) {
            atomicOr(a.status, SSM_STATUS_BAD_SLOT);
            ((T*)a.g)[(int64_t)b * a.E + c] = from_f32<T>(0.0f);
        }
        return;
    }
    *hp = make_float4(hn[0], hn[1], hn[2], hn[3]);
    if (q == 0) ((T*)a.g)[(int64_t)b * a.E + c] = from_f32<T>((y + Dc * u) * silu_f(z));
}

}  // namespace

// Window length: about target_windows(E) windows over the T tokens, so that every SIMD
// runs the same number of waves (the main pass fits 3 per SIMD). Any multiple of the
// token block works; rounding to a power of two instead left the busiest SIMDs a fifth
// more work than the average (2560 waves on 1024 SIMDs for the 2.8B half shard).
int scan_window_len(int64_t T, int E) {
    const int64_t tw = target_windows(E);
    const int64_t want = ((T + tw - 1) / tw + kTB - 1) / kTB * kTB;
    return (int)std::min<int64_t>(kMaxWin, std::max<int64_t>(kMinWin, want));
}

static int64_t max_windows(int64_t max_T, int E) {
    return std::max<int64_t>(target_windows(E), (max_T + kMaxWin - 1) / kMaxWin) + 1;
}

// Scratch regions of the windowed scan, in order: local end states [nwin][E][N],
// sums of Delta [nwin][E], linked entry states [nwin][E][N], copied initial states
// [nseq][E][N], window flags [nwin], Delta [T][E].
static size_t scan_layout(char* base, int64_t T, int E, int nseq, int nwin, ScanArgs* a, int32_t** wflags) {
    size_t off = 0;
    auto take = [&](size_t bytes) { char* p = base ? base + off : nullptr; off += align256(bytes); return p; };
    char* hl = take((size_t)nwin * E * kN * 4);
    char* sd = take((size_t)nwin * E * 4);
    char* hi = take((size_t)nwin * E * kN * 4);
    char* h0 = take((size_t)std::max(nseq, 1) * E * kN * 4);
    char* wf = take((size_t)std::max(nwin, 1) * 4);
    char* dl = take((size_t)std::max<int64_t>(T, 1) * E * 4);
    if (a) {
        a->h_local = (float*)hl; a->sum_delta = (float*)sd; a->h_in = (float*)hi; a->h0_seq = (float*)h0;
        a->delta = (float*)dl;
    }
    if (wflags) *wflags = (int32_t*)wf;
    return off;
}

static int num_windows(int64_t T, int win) { return T > 0 ? (int)((T + win - 1) / win) : 0; }

size_t scan_scratch_bytes(int64_t max_T, int E, int max_seqs) {
    // the window count is largest at the largest T (windows grow with T)
    const int nwin = std::max<int>((int)max_windows(max_T, E), num_windows(max_T, scan_window_len(max_T, E)));
    return scan_layout(nullptr, max_T, E, max_seqs, nwin, nullptr, nullptr);
}

hipError_t launch_scan_prefill(const ScanArgs& a0, bool bf, hipStream_t s) {
    ScanArgs a = a0;
    if (a.nseq <= 0) return hipSuccess;
    const int nwin = num_windows(a.T, a.win);
    int32_t* wflags = nullptr;
    scan_layout((char*)a0.h_local, a.T, a.E, a.nseq, nwin, &a, &wflags);
    const int cw = (a.E % (kWave * 4) == 0) ? 4 : 1;  // waves per workgroup sharing a window
    const dim3 grid((unsigned)(nwin * (a.E / (kWave * cw)))), block(kWave * cw);
    if (nwin > 0) {
        KernelTimer kt("prefill.scan_local", s);
        if (bf && cw == 4) SSM_LAUNCH((scan_local_kernel<bf16, 4>), grid, block, 0, s, a, nwin, wflags);
        else if (bf) SSM_LAUNCH((scan_local_kernel<bf16, 1>), grid, block, 0, s, a, nwin, wflags);
        else if (cw == 4) SSM_LAUNCH((scan_local_kernel<float, 4>), grid, block, 0, s, a, nwin, wflags);
        else SSM_LAUNCH((scan_local_kernel<float, 1>), grid, block, 0, s, a, nwin, wflags);
    }
    {
        KernelTimer kt("prefill.scan_link", s);
        const int64_t pairs = (int64_t)a.E * kN;
        SSM_LAUNCH(scan_link_kernel, dim3((unsigned)((pairs + kLinkPairs - 1) / kLinkPairs)),
                   dim3(kLinkSeg * kLinkPairs), 0, s, a, nwin,
                           (const int32_t*)wflags);
    }
    if (nwin > 0) {
        KernelTimer kt("prefill.scan_main", s);
        if (bf && cw == 4) SSM_LAUNCH((scan_main_kernel<bf16, 4>), grid, block, 0, s, a);
        else if (bf) SSM_LAUNCH((scan_main_kernel<bf16, 1>), grid, block, 0, s, a);
        else if (cw == 4) SSM_LAUNCH((scan_main_kernel<float, 4>), grid, block, 0, s, a);
        else SSM_LAUNCH((scan_main_kernel<float, 1>), grid, block, 0, s, a);
    }
    return hipGetLastError();
}

hipError_t launch_decode_ssm(const ScanArgs& a, bool bf, hipStream_t s) {
    const int64_t lanes = (int64_t)a.nseq * a.E * 4;
    if (lanes <= 0) return hipSuccess;
    const dim3 grid((unsigned)((lanes + 255) / 256)), block(256);
    if (bf) SSM_LAUNCH(decode_ssm_kernel<bf16>, grid, block, 0, s, a);
    else SSM_LAUNCH(decode_ssm_kernel<float>, grid, block, 0, s, a);
    return hipGetLastError();
}

}  // namespace ssm

namespace ssm {

hipError_t launch_decode_dt_ssm(const ScanArgs& a, bool bf, hipStream_t s) {
    if (a.nseq <= 0) return hipSuccess;
    if (a.R % 8 != 0 || a.E % kDtCh != 0 || a.ld_xdbl % 4 != 0 || ((uintptr_t)a.xdbl & 15) != 0 ||
        ((uintptr_t)a.w_dt & 15) != 0)
        return hipErrorNotSupported;
    if (bf && a.R % 32 == 0 && a.R <= 16 * 32) {
        // two 16-channel tiles per workgroup: E is a multiple of 64 (checked with the shape)
        constexpr int CT = 2;
        if (a.E % (CT * kDtCh) != 0) return hipErrorNotSupported;
        const dim3 g16((unsigned)(((a.nseq + kDtSeqM - 1) / kDtSeqM) * (a.E / (kDtCh * CT)))), b16(64 * kDtSeqM / kDtSpw);
        switch (a.R / 32) {
#define SSM_DTM(NK) case NK: SSM_LAUNCH((decode_dt_ssm_mfma_kernel<NK, kDtSpw, CT>), g16, b16, 0, s, a); break;
            SSM_DTM(1) SSM_DTM(2) SSM_DTM(3) SSM_DTM(4) SSM_DTM(5) SSM_DTM(6) SSM_DTM(7) SSM_DTM(8)
            SSM_DTM(9) SSM_DTM(10) SSM_DTM(11) SSM_DTM(12) SSM_DTM(13) SSM_DTM(14) SSM_DTM(15)
            default: SSM_LAUNCH((decode_dt_ssm_mfma_kernel<16, kDtSpw, CT>), g16, b16, 0, s, a); break;
#undef SSM_DTM
        }
        return hipGetLastError();
    }
    const dim3 grid((unsigned)(((a.nseq + kDtSeq - 1) / kDtSeq) * (a.E / kDtCh))), block(256);
    // chunks of 8 columns per lane: ceil(R / 32), R up to 256
    const int nch = (a.R / 8 + 3) / 4;
#define SSM_DTSSM(NC)                                                                            \
    if (bf) SSM_LAUNCH((decode_dt_ssm_kernel<bf16, NC>), grid, block, 0, s, a);                  \
    else SSM_LAUNCH((decode_dt_ssm_kernel<float, NC>), grid, block, 0, s, a);
    switch (nch) {
        case 1: SSM_DTSSM(1) break;
        case 2: SSM_DTSSM(2) break;
        case 3: SSM_DTSSM(3) break;
        case 4: SSM_DTSSM(4) break;
        case 5: SSM_DTSSM(5) break;
        case 6: SSM_DTSSM(6) break;
        case 7: SSM_DTSSM(7) break;
        case 8: SSM_DTSSM(8) break;
        default: return hipErrorNotSupported;  // dt_rank above 256: dt_proj and the state step apart
    }
#undef SSM_DTSSM
    return hipGetLastError();
}

}  // namespace ssm
