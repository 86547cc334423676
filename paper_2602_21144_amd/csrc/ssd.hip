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
// initial state; pass C: the full chunk walk from the linked state, writing g and the final
// state; then the per-head sums of g^2 for the gated norm.
#include <algorithm>

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

// bf16 row-major LDS tiles padded by 16 bytes per row: a fragment read of 16 consecutive rows
// at one column covers every bank once, and each access is a per-lane base plus a constant
constexpr int kLdS = kS + 8;   // row stride (elements) of a [rows][kS] tile
constexpr int kLdQ = kQ + 8;   // row stride of a [rows][kQ] tile

// one 32x32 MFMA tile: acc += A[rb.., k] * B[k, cb..] over k in [0, K), operands in LDS
// tiles A[row][k] (row stride LDA) and Bt[col][k] (row stride LDB)
template <int LDA, int LDB, int K>
__device__ __forceinline__ void mma_tile(f32x16& acc, const bf16* A, int rb, const bf16* Bt, int cb, int lane) {
    const int r = lane & 31, hk = (lane >> 5) * 8;
#pragma unroll
    for (int k0 = 0; k0 < K; k0 += 16) {
        const bf16x8 av = *(const bf16x8*)&A[(rb + r) * LDA + k0 + hk];
        const bf16x8 bv = *(const bf16x8*)&Bt[(cb + r) * LDB + k0 + hk];
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, bv, acc, 0, 0, 0);
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

// a plan entry is the same for the whole workgroup: keeping it in scalar registers keeps the
// buffer resources built from it scalar
__device__ __forceinline__ int4 uniform_plan(int4 p) {
    return make_int4(__builtin_amdgcn_readfirstlane(p.x), __builtin_amdgcn_readfirstlane(p.y),
                     __builtin_amdgcn_readfirstlane(p.z), __builtin_amdgcn_readfirstlane(p.w));
}

// ---------------------------------------------------------------- chunk machinery
// Wave w of a workgroup (0..3) holds the state rows n in [64 nh, 64 nh + 64), nh = w / 2, of
// the headdim block [pb, pb + 32), pb = 32 (w % 2), transposed, S^T[n][p], as two 32x32
// accumulator tiles; in pass C it also owns the output tile (headdim block pb, token block
// ib = 32 nh). A product whose contraction runs over the rows of an accumulator tile takes
// that tile as its operand directly: entries 8s..8s+7 of lane l are the rows
// 16s + 4 hh + {0..3} and 16s + 8 + 4 hh + {0..3} (hh = l / 32), which over both lane halves
// are the 16 contraction indices of one K-step, each once. The other operand is read from
// LDS in the same order, as two 8-byte pieces.

struct ChunkLds {
    bf16 Cs[kQ * kLdS];    // C      [i][n]
    bf16 Bs[kQ * kLdS];    // B      [j][n]
    bf16 Bt[kS * kLdQ];    // B^T    [n][j]
    bf16 Xt[kP * kLdQ];    // X^T    [p][j]
    float4 Zx[4][4][64];   // partial C S^T tile wave w hands to wave w ^ 2 (entry quad, lane)
    float cum[kQ], dl[kQ], wq[kQ];  // in-chunk cumulative log-decay, Delta, w
};

struct LocalLds {
    bf16 Bt[kS * kLdQ];
    bf16 Xt[kP * kLdQ];
    float cum[kQ], dl[kQ], wq[kQ];
};

// One chunk's inputs as this thread loads them for staging: B and X with the lane as the
// token (so that the transposing LDS writes of a wave are contiguous), C rows 16 B at a time,
// and (threads 0..63) one token's dt. Loads go through buffer resources over the chunk's
// valid rows, so rows past the chunk end read as zero without a branch.
struct ChunkRegs {
    bf16x8 b[4], c[4], x[2];
    float dt;
};

template <bool MAIN>
__device__ __forceinline__ void chunk_load(const SsdArgs& a, ChunkRegs& R, int h, int grp, int64_t t0, int nq) {
    const int tid = threadIdx.x, wave = tid >> 6, j = tid & 63;
    const __amdgpu_buffer_rsrc_t ru = buffer_rsrc(a.u + t0 * a.ld_u, (uint32_t)(nq * a.ld_u * 2));
    const __amdgpu_buffer_rsrc_t rz = buffer_rsrc(a.zx + t0 * a.ld_zx, (uint32_t)(nq * a.ld_zx * 2));
    const uint32_t row = (uint32_t)(j * a.ld_u);
#pragma unroll
    for (int it = 0; it < 4; ++it)   // B[j][n0 .. n0 + 8), n0 = 8 (wave + 4 it)
        R.b[it] = __builtin_bit_cast(bf16x8, buffer_load16(ru, (row + a.b_col + grp * kS + 8 * (wave + 4 * it)) * 2));
    if constexpr (MAIN) {
#pragma unroll
        for (int it = 0; it < 4; ++it) {   // C rows: 16 threads per row
            const int q = tid + kWG * it, jc = q >> 4, c8 = (q & 15) * 8;
            R.c[it] = __builtin_bit_cast(bf16x8, buffer_load16(ru, (uint32_t)(jc * a.ld_u + a.c_col + grp * kS + c8) * 2));
        }
    }
#pragma unroll
    for (int it = 0; it < 2; ++it)   // X[j][p0 .. p0 + 8), p0 = 8 (wave + 4 it)
        R.x[it] = __builtin_bit_cast(bf16x8, buffer_load16(ru, (row + h * kP + 8 * (wave + 4 * it)) * 2));
    const unsigned short dv = __builtin_amdgcn_raw_buffer_load_b16(
        rz, (int)((uint32_t)(j * a.ld_zx + a.dt_col + h) * 2), 0, 0);
    R.dt = (float)__builtin_bit_cast(bf16, dv);
}

// x and z of this lane's output entries (token ib + lane % 32, headdim pb + 8q + 4 hh + {0..3})
struct EpiRegs {
    bf16x4 x[4], z[4];
};

__device__ __forceinline__ void epi_load(const SsdArgs& a, EpiRegs& E, int h, int pb, int ib, int64_t t0, int nq,
                                         int lane) {
    const int i = ib + (lane & 31), c = h * kP + pb + 4 * (lane >> 5);
    const __amdgpu_buffer_rsrc_t ru = buffer_rsrc(a.u + t0 * a.ld_u, (uint32_t)(nq * a.ld_u * 2));
    const __amdgpu_buffer_rsrc_t rz = buffer_rsrc(a.zx + t0 * a.ld_zx, (uint32_t)(nq * a.ld_zx * 2));
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        E.x[q] = __builtin_bit_cast(bf16x4, __builtin_amdgcn_raw_buffer_load_b64(
                                                ru, (int)((uint32_t)(i * a.ld_u + c + 8 * q) * 2), 0, 0));
        E.z[q] = __builtin_bit_cast(bf16x4, __builtin_amdgcn_raw_buffer_load_b64(
                                                rz, (int)((uint32_t)(i * a.ld_zx + c + 8 * q) * 2), 0, 0));
    }
}

// registers -> LDS: B^T, X^T (and B, C); wave 0 turns dt into Delta, the in-chunk cumulative
// log-decay and w_j = exp(cum_last - cum_j) Delta_j (zero past the chunk end)
template <bool MAIN, class LDS>
__device__ __forceinline__ void chunk_put(LDS& L, const ChunkRegs& R, int nq, float A, float bias) {
    const int tid = threadIdx.x, wave = tid >> 6, j = tid & 63;
#pragma unroll
    for (int it = 0; it < 4; ++it) {
        const int n0 = 8 * (wave + 4 * it);
        if constexpr (MAIN) *(bf16x8*)&L.Bs[j * kLdS + n0] = R.b[it];
#pragma unroll
        for (int e = 0; e < 8; ++e) L.Bt[(n0 + e) * kLdQ + j] = R.b[it][e];
    }
    if constexpr (MAIN) {
#pragma unroll
        for (int it = 0; it < 4; ++it) {
            const int q = tid + kWG * it, jc = q >> 4, c8 = (q & 15) * 8;
            *(bf16x8*)&L.Cs[jc * kLdS + c8] = R.c[it];
        }
    }
#pragma unroll
    for (int it = 0; it < 2; ++it) {
        const int p0 = 8 * (wave + 4 * it);
#pragma unroll
        for (int e = 0; e < 8; ++e) L.Xt[(p0 + e) * kLdQ + j] = R.x[it][e];
    }
    if (tid < 64) {
        const float d = tid < nq ? softplus_dev(R.dt + bias) : 0.0f;
        float c = d * A;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const float o = __shfl_up(c, off, 64);
            if (tid >= off) c += o;
        }
        const float clast = __shfl(c, 63, 64);
        L.dl[tid] = d;
        L.cum[tid] = c;
        L.wq[tid] = __expf(clast - c) * d;
    }
}

// operand of one K-step read from a bf16 LDS tile: row r, contraction positions
// k0 + 4 hh + {0..3} and k0 + 8 + 4 hh + {0..3} (accumulator-row order)
template <int LD>
__device__ __forceinline__ bf16x8 perm_operand(const bf16* T, int r, int k0, int hh) {
    const bf16x4 lo = *(const bf16x4*)&T[r * LD + k0 + 4 * hh];
    const bf16x4 hi = *(const bf16x4*)&T[r * LD + k0 + 8 + 4 * hh];
    return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
}

// entries 8s..8s+7 of an accumulator tile as an operand: bf16 high part and remainder
__device__ __forceinline__ void acc_operand(const f32x16& acc, int s, bf16x8& hi, bf16x8& lo) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        const float v = acc[8 * s + e];
        const bf16 h = (bf16)v;
        hi[e] = h;
        lo[e] = (bf16)(v - (float)h);
    }
}

// S^T <- exp(cum_last) S^T + B^T (w o X) on this wave's two tiles; xa[s] is this lane's X^T
// operand of K-step s (row pb + lane % 32); w o X enters as high part and remainder
template <class LDS>
__device__ __forceinline__ void state_update(const LDS& L, f32x16 (&S)[2], const bf16x8 (&xa)[4], int nh, int lane) {
    const int r = lane & 31, hh = lane >> 5;
    const float dec = __expf(L.cum[kQ - 1]);
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int i = 0; i < 16; ++i) S[t][i] *= dec;
#pragma unroll
    for (int s = 0; s < 4; ++s) {
        const float4 w0 = *(const float4*)&L.wq[16 * s + 4 * hh];
        const float4 w1 = *(const float4*)&L.wq[16 * s + 8 + 4 * hh];
        const float wv[8] = {w0.x, w0.y, w0.z, w0.w, w1.x, w1.y, w1.z, w1.w};
        bf16x8 whi, wlo;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const float v = wv[e] * (float)xa[s][e];
            const bf16 h = (bf16)v;
            whi[e] = h;
            wlo[e] = (bf16)(v - (float)h);
        }
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            const bf16x8 bt = perm_operand<kLdQ>(L.Bt, 64 * nh + 32 * t + r, 16 * s, hh);
            S[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bt, whi, S[t], 0, 0, 0);
            S[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bt, wlo, S[t], 0, 0, 0);
        }
    }
}

// global state [P][N] fp32 <-> this wave's S^T tiles: entry 4q + b of tile t in lane l is
// p = pb + l % 32, n = 64 nh + 32 t + 8q + 4 hh + b
__device__ __forceinline__ void state_load(const float* src, f32x16 (&S)[2], int wave, int lane) {
    const int p = 32 * (wave & 1) + (lane & 31), n0 = 64 * (wave >> 1) + 4 * (lane >> 5);
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const float4 v = *(const float4*)&src[p * kS + n0 + 32 * t + 8 * q];
            S[t][4 * q] = v.x; S[t][4 * q + 1] = v.y; S[t][4 * q + 2] = v.z; S[t][4 * q + 3] = v.w;
        }
}

__device__ __forceinline__ void state_store(float* dst, const f32x16 (&S)[2], int wave, int lane) {
    const int p = 32 * (wave & 1) + (lane & 31), n0 = 64 * (wave >> 1) + 4 * (lane >> 5);
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int q = 0; q < 4; ++q)
            *(float4*)&dst[p * kS + n0 + 32 * t + 8 * q] =
                make_float4(S[t][4 * q], S[t][4 * q + 1], S[t][4 * q + 2], S[t][4 * q + 3]);
}

// ---------------------------------------------------------------- pass A
// Chunk c is staged from registers while chunk c+1's loads are in flight.
__global__ __launch_bounds__(kWG) __attribute__((amdgpu_waves_per_eu(4))) void ssd_local_kernel(SsdArgs a) {
    __shared__ LocalLds L;
    const int w = blockIdx.x, h = blockIdx.y;
    if (w >= *a.plan_count) return;
    const int4 pl = uniform_plan(a.plan[w]);
    if (pl.w & kWinLast) return;  // the last window's state is produced by pass C
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int nh = wave >> 1, pb = 32 * (wave & 1), r = lane & 31, hh = lane >> 5;
    const int grp = (a.h_global0 + h) / a.hpg - a.g_off;
    const float A = -__expf(a.A_log[h]), bias = a.dt_bias[h];
    f32x16 S[2] = {f32x16{}, f32x16{}};
    float lsum = 0.0f;
    ChunkRegs R;
    chunk_load<false>(a, R, h, grp, pl.y, rows_upto(pl.z - pl.y, kQ));
    for (int64_t t0 = pl.y; t0 < pl.z; t0 += kQ) {
        const int nq = rows_upto(pl.z - t0, kQ);
        chunk_put<false>(L, R, nq, A, bias);
        __syncthreads();
        if (t0 + kQ < pl.z) chunk_load<false>(a, R, h, grp, t0 + kQ, rows_upto(pl.z - t0 - kQ, kQ));
        bf16x8 xa[4];
#pragma unroll
        for (int s = 0; s < 4; ++s) xa[s] = perm_operand<kLdQ>(L.Xt, pb + r, 16 * s, hh);
        state_update(L, S, xa, nh, lane);
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
// Per chunk, wave (nh, pb) with token block ib = 32 nh:
//   Y^T[pb.., ib..] = X^T M^T over the causal j-blocks, M^T = (B C^T) o decay kept in registers
//   Z^T partials  = S C^T over its own state rows, for both token blocks; the one for the
//                   other block goes to wave w ^ 2 through LDS
//   S^T update (its own tiles), then after one barrier: g = (Y + exp(cum_i) Z + D x) SiLU(z)
// The next chunk's staging needs no barrier of its own: it only overwrites what all waves
// finished reading before the second barrier.
__global__ __launch_bounds__(kWG) __attribute__((amdgpu_waves_per_eu(2))) void ssd_main_kernel(SsdArgs a) {
    __shared__ ChunkLds L;
    const int w = blockIdx.x, h = blockIdx.y;
    if (w >= *a.plan_count) return;
    const int4 pl = uniform_plan(a.plan[w]);
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int nh = wave >> 1, pb = 32 * (wave & 1), ib = 32 * nh, r = lane & 31, hh = lane >> 5;
    const int grp = (a.h_global0 + h) / a.hpg - a.g_off;
    const float A = -__expf(a.A_log[h]), bias = a.dt_bias[h], Dh = a.D[h];
    f32x16 S[2];
    state_load(a.states + ((int64_t)w * a.H + h) * kP * kS, S, wave, lane);
    ChunkRegs R;
    EpiRegs Ep;
    {
        const int nq0 = rows_upto(pl.z - pl.y, kQ);
        chunk_load<true>(a, R, h, grp, pl.y, nq0);
        epi_load(a, Ep, h, pb, ib, pl.y, nq0, lane);
    }
    for (int64_t t0 = pl.y; t0 < pl.z; t0 += kQ) {
        const int nq = rows_upto(pl.z - t0, kQ);
        const bool more = t0 + kQ < pl.z;
        const int nqn = more ? rows_upto(pl.z - t0 - kQ, kQ) : 0;
        chunk_put<true>(L, R, nq, A, bias);
        __syncthreads();
        if (more) chunk_load<true>(a, R, h, grp, t0 + kQ, nqn);

        const int i = ib + r;
        const float ci = L.cum[i], eci = __expf(ci);
        bf16x8 xa[4];
#pragma unroll
        for (int s = 0; s < 4; ++s) xa[s] = perm_operand<kLdQ>(L.Xt, pb + r, 16 * s, hh);
        // Y^T = X^T M^T, M^T[j][i] = (B_j . C_i) exp(cum_i - cum_j) Delta_j for j <= i
        f32x16 Y = f32x16{};
#pragma unroll
        for (int jt = 0; jt < 2; ++jt) {
            if (32 * jt > ib) break;
            f32x16 G = f32x16{};
            mma_tile<kLdS, kLdS, kS>(G, L.Bs, 32 * jt, L.Cs, ib, lane);
            float m[16];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int j0 = 32 * jt + 8 * q + 4 * hh;
                const float4 cj = *(const float4*)&L.cum[j0];
                const float4 dj = *(const float4*)&L.dl[j0];
                const float cv[4] = {cj.x, cj.y, cj.z, cj.w}, dv[4] = {dj.x, dj.y, dj.z, dj.w};
#pragma unroll
                for (int b = 0; b < 4; ++b) {
                    // branch-free: the exponent is clamped (it is <= 0 wherever j <= i) and the
                    // causal mask selects Delta_j
                    const float ex = __expf(fminf(ci - cv[b], 0.0f));
                    m[4 * q + b] = G[4 * q + b] * ex * ((j0 + b <= i) ? dv[b] : 0.0f);
                }
            }
#pragma unroll
            for (int s = 0; s < 2; ++s) {
                bf16x8 mo;
#pragma unroll
                for (int e = 0; e < 8; ++e) mo[e] = (bf16)m[8 * s + e];
                Y = __builtin_amdgcn_mfma_f32_32x32x16_bf16(xa[2 * jt + s], mo, Y, 0, 0, 0);
            }
        }
        // Z^T partials over this wave's state rows, for token blocks 0 and 1
        f32x16 Zp[2] = {f32x16{}, f32x16{}};
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int s = 0; s < 2; ++s) {
                bf16x8 shi, slo;
                acc_operand(S[t], s, shi, slo);
#pragma unroll
                for (int ix = 0; ix < 2; ++ix) {
                    const bf16x8 cv = perm_operand<kLdS>(L.Cs, 32 * ix + r, 64 * nh + 32 * t + 16 * s, hh);
                    Zp[ix] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(shi, cv, Zp[ix], 0, 0, 0);
                    Zp[ix] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(slo, cv, Zp[ix], 0, 0, 0);
                }
            }
        {
            const f32x16& give = nh ? Zp[0] : Zp[1];
#pragma unroll
            for (int q = 0; q < 4; ++q)
                L.Zx[wave][q][lane] = make_float4(give[4 * q], give[4 * q + 1], give[4 * q + 2], give[4 * q + 3]);
        }
        state_update(L, S, xa, nh, lane);
        __syncthreads();

        // g = (Y + exp(cum_i) Z + D x) SiLU(z) for token t0 + i, headdim pb + 8q + 4 hh + {0..3}
        {
            const f32x16& own = nh ? Zp[1] : Zp[0];
            const __amdgpu_buffer_rsrc_t rg = buffer_rsrc(a.g + t0 * a.E, (uint32_t)(nq * a.E * 2));
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const float4 zo = L.Zx[wave ^ 2][q][lane];
                const float zv[4] = {zo.x, zo.y, zo.z, zo.w};
                bf16x4 gv;
#pragma unroll
                for (int b = 0; b < 4; ++b) {
                    const int e = 4 * q + b;
                    const float yv = Y[e] + eci * (own[e] + zv[b]) + Dh * (float)Ep.x[q][b];
                    gv[b] = (bf16)(yv * silu_f((float)Ep.z[q][b]));
                }
                __builtin_amdgcn_raw_buffer_store_b64(
                    __builtin_bit_cast(u32x2, gv), rg,
                    (int)((uint32_t)(i * a.E + h * kP + pb + 8 * q + 4 * hh) * 2), 0, 0);
            }
        }
        if (more) epi_load(a, Ep, h, pb, ib, t0 + kQ, nqn, lane);
    }
    if (pl.w & kWinLast) {
        const int slot = a.slot[pl.x];
        if (slot >= 0 && slot < a.S) state_store(a.pool + ((int64_t)slot * a.H + h) * kP * kS, S, wave, lane);
        else if (threadIdx.x == 0) atomicOr(a.status, SSM_STATUS_BAD_SLOT);
    }
}

// hs[t][h] = sum over the head's 64 channels of g^2: eight lanes per (token, head), each
// reading 16 consecutive bytes of the [T][H*64] tensor, so a wave reads 1 KB contiguously
__global__ __launch_bounds__(256) void ssd_head_sumsq_kernel(const bf16* __restrict__ g, int64_t n8,
                                                             float* __restrict__ hs) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;   // 8-element piece of g
    float s = 0.0f;
    if (i < n8) {
        const bf16x8 v = *(const bf16x8*)(g + i * 8);
#pragma unroll
        for (int e = 0; e < 8; ++e) s += (float)v[e] * (float)v[e];
    }
    s += __shfl_xor(s, 1, 64);
    s += __shfl_xor(s, 2, 64);
    s += __shfl_xor(s, 4, 64);
    if (i < n8 && (i & 7) == 0) hs[i >> 3] = s;
}

// ---------------------------------------------------------------- decode
// one workgroup per (sequence, head), 8 lanes per row p of the state: lane q holds the
// float4 groups at n = 32 j + 4 q (j = 0..3), so each load and store instruction of a wave
// covers 8 whole rows' 128-byte lines. Everything that does not depend on the cache slot
// (dt, x, z, the head's parameters, B_t, C_t) is fetched before the slot-addressed states.
__global__ __launch_bounds__(512) void ssd_decode_kernel(SsdArgs a) {
    const int b = blockIdx.x, h = blockIdx.y;
    const int tid = threadIdx.x, p = tid >> 3, q = tid & 7;
    __shared__ float ysq[8];
    const int slot = a.slot[b];
    const bf16* urow = a.u + (int64_t)b * a.ld_u;
    const bf16* zrow = a.zx + (int64_t)b * a.ld_zx;
    const int grp = (a.h_global0 + h) / a.hpg - a.g_off;
    const float dtv = (float)zrow[a.dt_col + h], zv = (float)zrow[h * kP + p];
    const float x = (float)urow[h * kP + p];
    const float dtb = a.dt_bias[h], alog = a.A_log[h], Dh = a.D[h];
    // B_t and C_t at this lane's n: 8-byte loads (b_col, c_col and ld_u are multiples of 8)
    bf16x4 bv[4], cv[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        bv[j] = *(const bf16x4*)(urow + a.b_col + grp * kS + 32 * j + 4 * q);
        cv[j] = *(const bf16x4*)(urow + a.c_col + grp * kS + 32 * j + 4 * q);
    }
    const bool ok = slot >= 0 && slot < a.S;
    // a slot outside the pool reads slot 0 (in range) and discards it
    float4* st = (float4*)(a.pool + (((int64_t)(ok ? slot : 0) * a.H + h) * kP + p) * kS) + q;
    float4 s4[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) s4[j] = st[8 * j];
    const float d = softplus_dev(dtv + dtb);
    const float dA = __expf(d * -__expf(alog)), dx = d * x;
    float acc = 0.0f;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        float sv[4] = {s4[j].x, s4[j].y, s4[j].z, s4[j].w};
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            sv[k] = dA * sv[k] + dx * (float)bv[j][k];
            acc += sv[k] * (float)cv[j][k];
        }
        s4[j] = make_float4(sv[0], sv[1], sv[2], sv[3]);
    }
    if (ok) {
#pragma unroll
        for (int j = 0; j < 4; ++j) st[8 * j] = s4[j];
    }
    acc += __shfl_xor(acc, 1, 64);
    acc += __shfl_xor(acc, 2, 64);
    acc += __shfl_xor(acc, 4, 64);
    const float y = acc + Dh * x;
    const bf16 gv = ok ? (bf16)(y * silu_f(zv)) : (bf16)0.0f;
    float sq = 0.0f;
    if (q == 0) {
        a.g[(int64_t)b * a.E + h * kP + p] = gv;
        sq = (float)gv * (float)gv;
    }
    sq += __shfl_xor(sq, 8, 64);
    sq += __shfl_xor(sq, 16, 64);
    sq += __shfl_xor(sq, 32, 64);
    if ((tid & 63) == 0) ysq[tid >> 6] = sq;
    __syncthreads();
    if (tid == 0) {
        float hsum = 0.0f;
#pragma unroll
        for (int w = 0; w < 8; ++w) hsum += ysq[w];
        a.hs[(int64_t)b * a.H + h] = hsum;
        if (!ok) atomicOr(a.status, SSM_STATUS_BAD_SLOT);
    }
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
    // the shard's heads in group k are the global heads [k hpg, (k + 1) hpg); blocks of 8
    // loads go out together and are added in ascending head order
    const int h0 = max(0, k * hpg - h_global0), h1 = min(H, (k + 1) * hpg - h_global0);
    const float* r = hs + t * H;
    float s = 0.0f;
    int h = h0;
    for (; h + 8 <= h1; h += 8) {
        float v[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = r[h + e];
#pragma unroll
        for (int e = 0; e < 8; ++e) s += v[e];
    }
    for (; h < h1; ++h) s += r[h];
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
    // about 1280 (window, head) workgroups: two and a half rounds of the 512 that are
    // resident at once (two per CU); windows are whole chunks, 64 to 2048 tokens
    const int64_t target = (1280 + H - 1) / H;
    const int64_t chunks = ((T + target - 1) / target + kQ - 1) / kQ;
    return (int)std::min<int64_t>(std::max<int64_t>(chunks, 1), 2048 / kQ) * kQ;
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
    {
        KernelTimer kt("prefill.ssd_head_sumsq", s);
        const int64_t n8 = p.T * a.H * (kP / 8);
        if (n8 > 0) SSM_LAUNCH(ssd_head_sumsq_kernel, dim3((unsigned)((n8 + 255) / 256)), dim3(256), 0, s, a.g, n8, a.hs);
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
    SSM_LAUNCH(ssd_decode_kernel, dim3((unsigned)batch, (unsigned)a.H), dim3(512), 0, s, a);
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
