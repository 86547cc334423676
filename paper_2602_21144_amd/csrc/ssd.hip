// Mamba-2 (SSD) state update of one shard (Section II-A: the state update reformulated so
// that it maps onto matrix products; Section IV-E: same pipeline and sharding as Mamba,
// per-head state, shard = a range of heads).
//
// Per head h (scalar decay A_h < 0, headdim P = 64, N = 128 states per row):
//   Delta_t = softplus(dt_t + dt_bias_h);  S_t = exp(Delta_t A_h) S_{t-1} + Delta_t x_t B_t^T
//   y_t = S_t C_t + D_h x_t;  g_t = y_t * SiLU(z_t)                         (S_t: P x N)
//
// Chunked form on MFMA, chunks of 64 tokens, cum_i = sum_{k<=i} Delta_k A_h within the chunk:
//   Y = M X + diag(exp(cum)) C S_in^T + D X,  M[i][j] = (C B^T)[i][j] exp(cum_i - cum_j) Delta_j (j <= i)
//   S_out = exp(cum_last) S_in + (w o X)^T B,  w_j = exp(cum_last - cum_j) Delta_j
// All four products are v_mfma_f32_32x32x16_bf16 with fp32 accumulation; the running state
// stays in the accumulators, and where it or w o X enters a product as an operand it is
// split into a bf16 high part and a bf16 remainder (two MFMAs) so that it keeps ~16 bits.
//
// Parallel layout: each sequence is cut into windows of whole chunks; a workgroup walks one
// (window, head) chunk by chunk. Pass A: each window's end state from zero (and its total
// log-decay); pass B: per state element, windows linked in order from the sequence's
// initial state; pass C: the full chunk walk from the linked state, writing g, the per-head
// sums of g^2 and the final state.
#include "common.h"

namespace ssm {
namespace {

constexpr int kQ = 64;    // tokens per chunk
constexpr int kP = 64;    // headdim
constexpr int kS = 128;   // d_state
constexpr int kWG = 256;  // threads per workgroup (4 waves)

// plan entry flags
constexpr int kWinFirst = 1, kWinLast = 2;

__device__ __forceinline__ float softplus_dev(float v) { return softplus_f(v); }

// bf16 row-major LDS tiles with 16-byte chunks XOR-permuted by row, so that the 32 rows a
// fragment read touches spread over the banks
template <int COLS> __device__ __forceinline__ int toff(int row, int col) {
    constexpr int KC = COLS / 8;
    static_assert(KC >= 8 && (KC & (KC - 1)) == 0, "power-of-two chunk count");
    return row * COLS + ((((col >> 3) ^ (row & 7))) << 3) + (col & 7);
}

// one 32x32 MFMA tile: acc += A[rb.., k] * B[k, cb..] over k in [0, K), operands in LDS
// tiles A[row][k] (COLS_A wide) and Bt[col][k] (COLS_B wide)
template <int COLS_A, int COLS_B, int K>
__device__ __forceinline__ void mma_tile(f32x16& acc, const bf16* A, int rb, const bf16* Bt, int cb, int lane) {
    const int r = lane & 31, hk = (lane >> 5) * 8;
#pragma unroll
    for (int k0 = 0; k0 < K; k0 += 16) {
        const bf16x8 a = *(const bf16x8*)&A[toff<COLS_A>(rb + r, k0 + hk)];
        const bf16x8 b = *(const bf16x8*)&Bt[toff<COLS_B>(cb + r, k0 + hk)];
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc, 0, 0, 0);
    }
}

// element (row, col) of accumulator entry i in lane l of a 32x32 tile at (rb, cb)
__device__ __forceinline__ int acc_row(int rb, int i, int lane) { return rb + 8 * (i >> 2) + 4 * (lane >> 5) + (i & 3); }
__device__ __forceinline__ int acc_col(int cb, int lane) { return cb + (lane & 31); }

struct SsdArgs {
    const bf16* zx;   int64_t ld_zx;   // in_proj output [T][ld_zx]: z at col 0, dt at col dt_col
    const bf16* u;    int64_t ld_u;    // conv output [T][ld_u]: x at col 0, B at b_col, C at c_col
    int dt_col, b_col, c_col;
    int H, E;                          // heads of the shard, E = H * P
    int h_global0, hpg, g_off;         // head h is global head h_global0 + h; its B/C group is
                                       // (h_global0 + h) / hpg, stored at local group index - g_off
    const float* dt_bias; const float* A_log; const float* D;
    bf16* g;                           // [T][E]
    float* hs;                         // [T][H] sum over the head's channels of g^2
    float* pool;                       // [S][H][P][N]
    const int32_t* cu; const int32_t* slot; const int32_t* has_init;
    int32_t* status;
    int nseq, S, win;
    int64_t T;                         // packed tokens (the plan never reaches past it)
    int4* plan; int32_t* plan_count; int max_windows;
    float* states;                     // [max_windows][H][P][N]
    float* lsum;                       // [max_windows][H] total log-decay of the window
};

// ---------------------------------------------------------------- window plan
__global__ void ssd_plan_kernel(SsdArgs a) {
    if (threadIdx.x != 0) return;
    int w = 0;
    bool bad = false;
    for (int s = 0; s < a.nseq; ++s) {
        const int b = a.cu[s], e = a.cu[s + 1];
        if (b < 0 || e < b || e > a.T) { bad = true; continue; }
        const int nw = (e - b + a.win - 1) / a.win;
        for (int k = 0; k < nw && w < a.max_windows; ++k, ++w) {
            const int t0 = b + k * a.win, t1 = min(t0 + a.win, e);
            a.plan[w] = make_int4(s, t0, t1, (k == 0 ? kWinFirst : 0) | (k == nw - 1 ? kWinLast : 0));
        }
    }
    *a.plan_count = w;
    if (bad) atomicOr(a.status, SSM_STATUS_BAD_SEQLENS);
}

// ---------------------------------------------------------------- chunk machinery
struct ChunkLds {
    bf16 Cs[kQ * kS];      // C      [i][n]
    bf16 Bs[kQ * kS];      // B      [j][n]
    bf16 Bt[kS * kQ];      // B^T    [n][j]
    bf16 Xt[kP * kQ];      // X^T    [p][j]
    bf16 Wh[kP * kQ];      // (w o X)^T high part [p][j]
    bf16 Wl[kP * kQ];      // remainder
    bf16 Ms[kQ * kQ];      // M      [i][j]
    bf16 Zs[kQ * kP];      // z      [i][p]
    bf16 Sh[kP * kS];      // state high part [p][n]
    bf16 Sl[kP * kS];      // remainder
    float cum[kQ], dl[kQ], rowsq[2][kQ];
};

__device__ __forceinline__ void split_bf16(float v, bf16& hi, bf16& lo) {
    hi = (bf16)v;
    lo = (bf16)(v - (float)hi);
}

// Delta and the in-chunk cumulative log-decay (wave 0: one lane per token)
__device__ __forceinline__ void chunk_decay(const SsdArgs& a, ChunkLds& L, int h, int64_t t0, int nq, float A, float bias) {
    const int lane = threadIdx.x;
    if (lane >= 64) return;
    float d = 0.0f;
    if (lane < nq) d = softplus_dev((float)a.zx[(t0 + lane) * a.ld_zx + a.dt_col + h] + bias);
    float c = d * A;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const float o = __shfl_up(c, off, 64);
        if (lane >= off) c += o;
    }
    L.dl[lane] = d;
    L.cum[lane] = c;
}

// stage B (both layouts) and X^T, and with the decay known the split (w o X)^T
template <bool WITH_C>
__device__ __forceinline__ void chunk_stage(const SsdArgs& a, ChunkLds& L, int h, int64_t t0, int nq) {
    const int tid = threadIdx.x;
    const int grp = (a.h_global0 + h) / a.hpg - a.g_off;
    // B and C: 64 rows x 128 columns, 16 columns (32 B) per thread-step
    for (int q = tid; q < kQ * (kS / 8); q += kWG) {
        const int j = q / (kS / 8), c8 = (q % (kS / 8)) * 8;
        bf16x8 bv = bf16x8{}, cv = bf16x8{};
        if (j < nq) {
            const bf16* row = a.u + (t0 + j) * a.ld_u;
            bv = *(const bf16x8*)(row + a.b_col + grp * kS + c8);
            if constexpr (WITH_C) cv = *(const bf16x8*)(row + a.c_col + grp * kS + c8);
        }
        *(bf16x8*)&L.Bs[toff<kS>(j, c8)] = bv;
        if constexpr (WITH_C) *(bf16x8*)&L.Cs[toff<kS>(j, c8)] = cv;
#pragma unroll
        for (int e = 0; e < 8; ++e) L.Bt[toff<kQ>(c8 + e, j)] = bv[e];
    }
    const float clast = L.cum[kQ - 1];
    for (int q = tid; q < kQ * (kP / 8); q += kWG) {
        const int j = q / (kP / 8), p8 = (q % (kP / 8)) * 8;
        bf16x8 xv = bf16x8{}, zv = bf16x8{};
        if (j < nq) {
            xv = *(const bf16x8*)(a.u + (t0 + j) * a.ld_u + h * kP + p8);
            if constexpr (WITH_C) zv = *(const bf16x8*)(a.zx + (t0 + j) * a.ld_zx + h * kP + p8);
        }
        if constexpr (WITH_C) *(bf16x8*)&L.Zs[toff<kP>(j, p8)] = zv;
        const float wj = j < nq ? __expf(clast - L.cum[j]) * L.dl[j] : 0.0f;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            L.Xt[toff<kQ>(p8 + e, j)] = xv[e];
            bf16 hi, lo;
            split_bf16(wj * (float)xv[e], hi, lo);
            L.Wh[toff<kQ>(p8 + e, j)] = hi;
            L.Wl[toff<kQ>(p8 + e, j)] = lo;
        }
    }
}

// S (this wave's two 32x32 tiles of the P x N state) <- exp(cum_last) S + (w o X)^T B
__device__ __forceinline__ void chunk_state_update(ChunkLds& L, f32x16 (&S)[2], int wave, int lane) {
    const float dec = __expf(L.cum[kQ - 1]);
    const int pb = (wave >> 1) * 32;
#pragma unroll
    for (int t = 0; t < 2; ++t) {
        const int nb = ((wave & 1) * 2 + t) * 32;
#pragma unroll
        for (int i = 0; i < 16; ++i) S[t][i] *= dec;
        mma_tile<kQ, kQ, kQ>(S[t], L.Wh, pb, L.Bt, nb, lane);
        mma_tile<kQ, kQ, kQ>(S[t], L.Wl, pb, L.Bt, nb, lane);
    }
}

__device__ __forceinline__ void state_to_lds(ChunkLds& L, const f32x16 (&S)[2], int wave, int lane) {
    const int pb = (wave >> 1) * 32;
#pragma unroll
    for (int t = 0; t < 2; ++t) {
        const int nb = ((wave & 1) * 2 + t) * 32;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            bf16 hi, lo;
            split_bf16(S[t][i], hi, lo);
            const int p = acc_row(pb, i, lane), n = acc_col(nb, lane);
            L.Sh[toff<kS>(p, n)] = hi;
            L.Sl[toff<kS>(p, n)] = lo;
        }
    }
}

__device__ __forceinline__ void state_load(const float* src, f32x16 (&S)[2], int wave, int lane) {
    const int pb = (wave >> 1) * 32;
#pragma unroll
    for (int t = 0; t < 2; ++t) {
        const int nb = ((wave & 1) * 2 + t) * 32;
#pragma unroll
        for (int i = 0; i < 16; ++i) S[t][i] = src[acc_row(pb, i, lane) * kS + acc_col(nb, lane)];
    }
}

__device__ __forceinline__ void state_store(float* dst, const f32x16 (&S)[2], int wave, int lane) {
    const int pb = (wave >> 1) * 32;
#pragma unroll
    for (int t = 0; t < 2; ++t) {
        const int nb = ((wave & 1) * 2 + t) * 32;
#pragma unroll
        for (int i = 0; i < 16; ++i) dst[acc_row(pb, i, lane) * kS + acc_col(nb, lane)] = S[t][i];
    }
}

// ---------------------------------------------------------------- pass A
__global__ __launch_bounds__(kWG) void ssd_local_kernel(SsdArgs a) {
    __shared__ ChunkLds L;
    const int w = blockIdx.x, h = blockIdx.y;
    if (w >= *a.plan_count) return;
    const int4 pl = a.plan[w];
    if (pl.w & kWinLast) return;  // the last window's state is produced by pass C
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const float A = -__expf(a.A_log[h]), bias = a.dt_bias[h];
    f32x16 S[2] = {f32x16{}, f32x16{}};
    float lsum = 0.0f;
    for (int64_t t0 = pl.y; t0 < pl.z; t0 += kQ) {
        const int nq = (int)min<int64_t>(kQ, pl.z - t0);
        chunk_decay(a, L, h, t0, nq, A, bias);
        __syncthreads();
        chunk_stage<false>(a, L, h, t0, nq);
        __syncthreads();
        chunk_state_update(L, S, wave, lane);
        lsum += L.cum[kQ - 1];
        __syncthreads();
    }
    state_store(a.states + ((int64_t)w * a.H + h) * kP * kS, S, wave, lane);
    if (threadIdx.x == 0) a.lsum[(int64_t)w * a.H + h] = lsum;
}

// ---------------------------------------------------------------- pass B
// one lane per (head, p, n): walk the windows in plan order
__global__ __launch_bounds__(256) void ssd_link_kernel(SsdArgs a) {
    const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (gid >= (int64_t)a.H * kP * kS) return;
    const int h = (int)(gid / (kP * kS));
    const int e = (int)(gid % (kP * kS));
    const int nw = *a.plan_count;
    float carry = 0.0f;
    for (int w = 0; w < nw; ++w) {
        const int4 pl = a.plan[w];
        if (pl.w & kWinFirst) {
            carry = 0.0f;
            if (a.has_init[pl.x]) {
                const int slot = a.slot[pl.x];
                if (slot >= 0 && slot < a.S) carry = a.pool[((int64_t)slot * a.H + h) * kP * kS + e];
                else if (e == 0) atomicOr(a.status, SSM_STATUS_BAD_SLOT);
            }
        }
        float* st = a.states + ((int64_t)w * a.H + h) * kP * kS + e;
        const float local = (pl.w & kWinLast) ? 0.0f : *st;
        *st = carry;  // state entering the window
        if (!(pl.w & kWinLast)) carry = __expf(a.lsum[(int64_t)w * a.H + h]) * carry + local;
    }
    // empty sequences that start fresh end with a zero state
    for (int s = 0; s < a.nseq; ++s) {
        if (a.cu[s + 1] != a.cu[s] || a.has_init[s]) continue;
        const int slot = a.slot[s];
        if (slot >= 0 && slot < a.S) a.pool[((int64_t)slot * a.H + h) * kP * kS + e] = 0.0f;
    }
}

// ---------------------------------------------------------------- pass C
__global__ __launch_bounds__(kWG) void ssd_main_kernel(SsdArgs a) {
    __shared__ ChunkLds L;
    const int w = blockIdx.x, h = blockIdx.y;
    if (w >= *a.plan_count) return;
    const int4 pl = a.plan[w];
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const float A = -__expf(a.A_log[h]), bias = a.dt_bias[h], Dh = a.D[h];
    f32x16 S[2];
    state_load(a.states + ((int64_t)w * a.H + h) * kP * kS, S, wave, lane);
    state_to_lds(L, S, wave, lane);
    // this wave's 32x32 tile of the chunk output Y [i][p]
    const int rb = (wave >> 1) * 32, cb = (wave & 1) * 32;
    for (int64_t t0 = pl.y; t0 < pl.z; t0 += kQ) {
        const int nq = (int)min<int64_t>(kQ, pl.z - t0);
        chunk_decay(a, L, h, t0, nq, A, bias);
        __syncthreads();
        chunk_stage<true>(a, L, h, t0, nq);
        __syncthreads();
        // M = (C B^T) o decay mask, written as bf16 [i][j]
        {
            f32x16 G = f32x16{};
            mma_tile<kS, kS, kS>(G, L.Cs, rb, L.Bs, cb, lane);
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int r = acc_row(rb, i, lane), c = acc_col(cb, lane);
                const float m = (c <= r && r < nq) ? G[i] * __expf(L.cum[r] - L.cum[c]) * L.dl[c] : 0.0f;
                L.Ms[toff<kQ>(r, c)] = (bf16)m;
            }
        }
        // C S_in^T (state entering this chunk), before the barrier lets anyone overwrite Sh/Sl
        f32x16 Z = f32x16{};
        mma_tile<kS, kS, kS>(Z, L.Cs, rb, L.Sh, cb, lane);
        mma_tile<kS, kS, kS>(Z, L.Cs, rb, L.Sl, cb, lane);
        __syncthreads();
        f32x16 Y = f32x16{};
        mma_tile<kQ, kQ, kQ>(Y, L.Ms, rb, L.Xt, cb, lane);
        float sq[16];
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            const int r = acc_row(rb, i, lane), c = acc_col(cb, lane);
            const float x = (float)L.Xt[toff<kQ>(c, r)];
            const float yv = Y[i] + __expf(L.cum[r]) * Z[i] + Dh * x;
            const bf16 gv = (bf16)(yv * silu_f((float)L.Zs[toff<kP>(r, c)]));
            if (r < nq) a.g[(t0 + r) * a.E + h * kP + c] = gv;
            const float gf = (float)gv;
            sq[i] = gf * gf;
        }
        // sum of g^2 over this tile's 32 columns for each of its rows, then over the two
        // column tiles of the head
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            float v = sq[i];
#pragma unroll
            for (int off = 16; off >= 1; off >>= 1) v += __shfl_xor(v, off, 32);
            sq[i] = v;
        }
        if ((lane & 31) == 0) {
#pragma unroll
            for (int i = 0; i < 16; ++i) L.rowsq[wave & 1][acc_row(rb, i, lane)] = sq[i];
        }
        chunk_state_update(L, S, wave, lane);
        __syncthreads();
        if (threadIdx.x < nq) a.hs[(t0 + threadIdx.x) * a.H + h] = L.rowsq[0][threadIdx.x] + L.rowsq[1][threadIdx.x];
        state_to_lds(L, S, wave, lane);
        __syncthreads();
    }
    if (pl.w & kWinLast) {
        const int slot = a.slot[pl.x];
        if (slot >= 0 && slot < a.S) state_store(a.pool + ((int64_t)slot * a.H + h) * kP * kS, S, wave, lane);
        else if (threadIdx.x == 0) atomicOr(a.status, SSM_STATUS_BAD_SLOT);
    }
}

// ---------------------------------------------------------------- decode
// one workgroup per (sequence, head): 4 lanes per row p of the state, 32 states each
__global__ __launch_bounds__(256) void ssd_decode_kernel(SsdArgs a, int batch) {
    const int b = blockIdx.x, h = blockIdx.y;
    const int tid = threadIdx.x, p = tid >> 2, n0 = (tid & 3) * 32;
    __shared__ float ysq[4];
    const int slot = a.slot[b];
    const bool ok = slot >= 0 && slot < a.S;
    const bf16* urow = a.u + (int64_t)b * a.ld_u;
    const int grp = (a.h_global0 + h) / a.hpg - a.g_off;
    const float d = softplus_dev((float)a.zx[(int64_t)b * a.ld_zx + a.dt_col + h] + a.dt_bias[h]);
    const float dA = __expf(d * -__expf(a.A_log[h]));
    const float x = (float)urow[h * kP + p];
    float* st = a.pool + (((int64_t)(ok ? slot : 0) * a.H + h) * kP + p) * kS + n0;
    float acc = 0.0f;
#pragma unroll
    for (int q = 0; q < 32; q += 4) {
        float4 s4 = ok ? *(const float4*)(st + q) : make_float4(0.f, 0.f, 0.f, 0.f);
        float sv[4] = {s4.x, s4.y, s4.z, s4.w};
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int n = n0 + q + k;
            sv[k] = dA * sv[k] + d * x * (float)urow[a.b_col + grp * kS + n];
            acc += sv[k] * (float)urow[a.c_col + grp * kS + n];
        }
        if (ok) *(float4*)(st + q) = make_float4(sv[0], sv[1], sv[2], sv[3]);
    }
    acc += __shfl_xor(acc, 1, 64);
    acc += __shfl_xor(acc, 2, 64);
    const float y = acc + a.D[h] * x;
    const bf16 gv = ok ? (bf16)(y * silu_f((float)a.zx[(int64_t)b * a.ld_zx + h * kP + p])) : (bf16)0.0f;
    float sq = 0.0f;
    if ((tid & 3) == 0) {
        a.g[(int64_t)b * a.E + h * kP + p] = gv;
        sq = (float)gv * (float)gv;
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) sq += __shfl_xor(sq, off, 64);
    if ((tid & 63) == 0) ysq[tid >> 6] = sq;
    __syncthreads();
    if (tid == 0) {
        a.hs[(int64_t)b * a.H + h] = ysq[0] + ysq[1] + ysq[2] + ysq[3];
        if (!ok) atomicOr(a.status, SSM_STATUS_BAD_SLOT);
    }
    (void)batch;
}

// ---------------------------------------------------------------- norm
// out[t][k] = sum over the shard's heads in norm group k of hs[t][h] (fixed order)
// (the norm group of a head is its global B/C group: both span nheads / ngroups heads)
__global__ __launch_bounds__(256) void ssd_group_sumsq_kernel(const float* __restrict__ hs, int H, int h_global0,
                                                              int hpg, int G, float* __restrict__ out, int64_t T) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= T * G) return;
    const int64_t t = i / G;
    const int k = (int)(i % G);
    float s = 0.0f;
    for (int h = 0; h < H; ++h)
        if ((h_global0 + h) / hpg == k) s += hs[t * H + h];
    out[i] = s;
}

// gn[t][c] = bf16(g[t][c] / sqrt(sumsq[t][k(c)] / gsize + eps) * norm_w[c]), 8 channels per thread
__global__ __launch_bounds__(256) void ssd_norm_kernel(const bf16* __restrict__ g, const float* __restrict__ sumsq,
                                                       const float* __restrict__ norm_w, bf16* __restrict__ out,
                                                       int64_t T, int E, int G, int gsize, int c_global0, float eps) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const int per = E / 8;
    if (i >= T * per) return;
    const int64_t t = i / per;
    const int c = (int)(i % per) * 8;
    const int k = (c_global0 + c) / gsize;
    const float inv = 1.0f / sqrtf(sumsq[t * G + k] / (float)gsize + eps);
    const bf16x8 v = *(const bf16x8*)(g + t * E + c);
    bf16x8 o;
#pragma unroll
    for (int e = 0; e < 8; ++e) o[e] = (bf16)((float)v[e] * inv * norm_w[c + e]);
    *(bf16x8*)(out + t * E + c) = o;
}

}  // namespace

int ssd_window_len(int64_t T, int H) {
    // enough (window, head) workgroups to fill the chip a few times over
    int64_t target = (4 * 256 + H - 1) / H;
    int64_t win = (T + target - 1) / target;
    int w = kQ;
    while (w < win && w < 2048) w <<= 1;
    return w;
}

int ssd_max_windows(int64_t T, int nseq, int win) { return (int)((T + win - 1) / win + nseq); }

size_t ssd_state_bytes(int max_windows, int H) { return (size_t)max_windows * H * kP * kS * 4; }

hipError_t launch_ssd_prefill(const SsdPublic& p, hipStream_t s) {
    SsdArgs a{};
    a.zx = (const bf16*)p.zx; a.ld_zx = p.ld_zx; a.u = (const bf16*)p.u; a.ld_u = p.ld_u;
    a.dt_col = p.dt_col; a.b_col = p.b_col; a.c_col = p.c_col; a.H = p.H; a.E = p.H * kP;
    a.h_global0 = p.h_global0; a.hpg = p.hpg; a.g_off = p.g_off;
    a.dt_bias = p.dt_bias; a.A_log = p.A_log; a.D = p.D;
    a.g = (bf16*)p.g; a.hs = p.hs; a.pool = p.pool; a.cu = p.cu; a.slot = p.slot; a.has_init = p.has_init;
    a.status = p.status; a.nseq = p.nseq; a.S = p.S; a.win = p.win; a.T = p.T; a.plan = (int4*)p.plan;
    a.plan_count = p.plan_count; a.max_windows = p.max_windows; a.states = p.states; a.lsum = p.lsum;
    if (a.nseq <= 0) return hipSuccess;
    {
        KernelTimer kt("prefill.ssd_plan", s);
        SSM_LAUNCH(ssd_plan_kernel, dim3(1), dim3(64), 0, s, a);
    }
    const dim3 grid((unsigned)a.max_windows, (unsigned)a.H);
    {
        KernelTimer kt("prefill.ssd_local", s);
        SSM_LAUNCH(ssd_local_kernel, grid, dim3(kWG), 0, s, a);
    }
    {
        KernelTimer kt("prefill.ssd_link", s);
        const int64_t lanes = (int64_t)a.H * kP * kS;
        SSM_LAUNCH(ssd_link_kernel, dim3((unsigned)((lanes + 255) / 256)), dim3(256), 0, s, a);
    }
    {
        KernelTimer kt("prefill.ssd_main", s);
        SSM_LAUNCH(ssd_main_kernel, grid, dim3(kWG), 0, s, a);
    }
    return hipGetLastError();
}

hipError_t launch_ssd_decode(const SsdPublic& p, int batch, hipStream_t s) {
    if (batch <= 0) return hipSuccess;
    SsdArgs a{};
    a.zx = (const bf16*)p.zx; a.ld_zx = p.ld_zx; a.u = (const bf16*)p.u; a.ld_u = p.ld_u;
    a.dt_col = p.dt_col; a.b_col = p.b_col; a.c_col = p.c_col; a.H = p.H; a.E = p.H * kP;
    a.h_global0 = p.h_global0; a.hpg = p.hpg; a.g_off = p.g_off;
    a.dt_bias = p.dt_bias; a.A_log = p.A_log; a.D = p.D;
    a.g = (bf16*)p.g; a.hs = p.hs; a.pool = p.pool; a.slot = p.slot; a.status = p.status; a.S = p.S;
    SSM_LAUNCH(ssd_decode_kernel, dim3((unsigned)batch, (unsigned)a.H), dim3(256), 0, s, a, batch);
    return hipGetLastError();
}

hipError_t launch_ssd_group_sumsq(const float* hs, int H, int h_global0, int hpg, int G, float* out, int64_t T,
                                  hipStream_t s) {
    if (T <= 0) return hipSuccess;
    SSM_LAUNCH(ssd_group_sumsq_kernel, dim3((unsigned)((T * G + 255) / 256)), dim3(256), 0, s, hs, H, h_global0, hpg,
               G, out, T);
    return hipGetLastError();
}

hipError_t launch_ssd_norm(const void* g, const float* sumsq, const float* norm_w, void* out, int64_t T, int E, int G,
                           int gsize, int c_global0, float eps, hipStream_t s) {
    if (T <= 0) return hipSuccess;
    SSM_LAUNCH(ssd_norm_kernel, dim3((unsigned)((T * (E / 8) + 255) / 256)), dim3(256), 0, s, (const bf16*)g, sumsq,
               norm_w, (bf16*)out, T, E, G, gsize, c_global0, eps);
    return hipGetLastError();
}

}  // namespace ssm
