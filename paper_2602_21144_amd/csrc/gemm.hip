// Dense projections of the mixer (in_proj, x_proj, dt_proj, out_proj) as
// C[M][N] = A[M][K] * B[N][K]^T on gfx950 matrix cores.
//
// Both operands are K-contiguous (activations [tokens][features], weights
// [out_features][in_features]), which is the natural operand layout of MFMA: every
// lane loads 8 consecutive k of one row. bf16 path: v_mfma_f32_32x32x16_bf16 with
// fp32 accumulation; fp32 path: v_mfma_f32_16x16x4_f32.
#include <algorithm>
#include <type_traits>
#include <utility>

#include "common.h"

namespace ssm {
namespace {

constexpr int kBK = 64;  // k per LDS stage (bf16): 128 bytes per row = 8 chunks of 16 B

// Row r of an LDS tile stores its 8 chunks permuted by an XOR with (r>>1)&7, so the
// 16 lanes that read one chunk column from 16 consecutive rows hit distinct banks.
__device__ __forceinline__ int swz(int row, int chunk) { return chunk ^ ((row >> 1) & 7); }

// Map the linear workgroup id to an output tile. Workgroups are dispatched round robin
// over the 8 XCDs; regroup so each XCD gets a contiguous run of tiles, and order the
// tiles in groups of 4 tile-rows so that a run shares A panels and B panels in its L2
// (groups of 4 took dt_proj's 2560 short tiles from 31 to 28 us; 8 and 16 measured the
// same or slower on every projection).
__device__ __forceinline__ void tile_of(int tiles_m, int tiles_n, int& tm, int& tn) {
    int nwg = gridDim.x;
    int bid = blockIdx.x;
    if ((nwg & 7) == 0) bid = (bid & 7) * (nwg >> 3) + (bid >> 3);
    constexpr int G = 4;
    int per_group = G * tiles_n;
    int grp = bid / per_group;
    int first = grp * G;
    int gm = min(tiles_m - first, G);
    int r = bid - grp * per_group;
    tm = first + r % gm;
    tn = r / gm;
}

__device__ __forceinline__ bf16x8 cvt8(float4 a, float4 b) {
    bf16x8 o;
    o[0] = (bf16)a.x; o[1] = (bf16)a.y; o[2] = (bf16)a.z; o[3] = (bf16)a.w;
    o[4] = (bf16)b.x; o[5] = (bf16)b.y; o[6] = (bf16)b.z; o[7] = (bf16)b.w;
    return o;
}

// ROLE only names the instance (one kernel symbol per projection, so profiles separate them).
template <int ROLE, int BM, int BN, int WM, int WN, bool A_F32, bool C_F32>
__global__ __launch_bounds__(256) void gemm_bf16_nt(int M, int N, int K,
                                                    const void* __restrict__ Ap, int64_t lda,
                                                    const bf16* __restrict__ B, int64_t ldb,
                                                    void* __restrict__ Cp, int64_t ldc,
                                                    int tiles_m, int tiles_n) {
    static_assert(WM * WN == 4, "four waves");
    constexpr int WTM = BM / WM, WTN = BN / WN;
    constexpr int TM = WTM / 32, TN = WTN / 32;
    static_assert(TM >= 1 && TN >= 1 && WTM % 32 == 0 && WTN % 32 == 0, "wave tile");
    constexpr int AC = BM * 8 / 256;  // 16-byte chunks per thread per stage
    constexpr int BC = BN * 8 / 256;
    static_assert(AC >= 1 && BC >= 1, "tile too small for 256 threads");

    __shared__ __attribute__((aligned(16))) bf16 As[2][BM * kBK];
    __shared__ __attribute__((aligned(16))) bf16 Bs[2][BN * kBK];

    int tm, tn;
    tile_of(tiles_m, tiles_n, tm, tn);
    const int m0 = tm * BM, n0 = tn * BN;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave / WN, wn = wave % WN;

    bf16x8 ra[AC], rb[BC];

    auto gload = [&](int k0) {
#pragma unroll
        for (int i = 0; i < AC; ++i) {
            const int q = tid + 256 * i, row = q >> 3, ck = q & 7;
            const int gm = m0 + row, gk = k0 + ck * 8;
            if (gm < M && gk < K) {
                if constexpr (A_F32) {
                    const float* p = (const float*)Ap + (int64_t)gm * lda + gk;
                    ra[i] = cvt8(*(const float4*)p, *(const float4*)(p + 4));
                } else {
                    ra[i] = *(const bf16x8*)((const bf16*)Ap + (int64_t)gm * lda + gk);
                }
            } else {
                ra[i] = bf16x8{};
            }
        }
#pragma unroll
        for (int i = 0; i < BC; ++i) {
            const int q = tid + 256 * i, row = q >> 3, ck = q & 7;
            const int gn = n0 + row, gk = k0 + ck * 8;
            rb[i] = (gn < N && gk < K) ? *(const bf16x8*)(B + (int64_t)gn * ldb + gk) : bf16x8{};
        }
    };
    auto lstore = [&](int buf) {
#pragma unroll
        for (int i = 0; i < AC; ++i) {
            const int q = tid + 256 * i, row = q >> 3, ck = q & 7;
            *(bf16x8*)&As[buf][row * kBK + swz(row, ck) * 8] = ra[i];
        }
#pragma unroll
        for (int i = 0; i < BC; ++i) {
            const int q = tid + 256 * i, row = q >> 3, ck = q & 7;
            *(bf16x8*)&Bs[buf][row * kBK + swz(row, ck) * 8] = rb[i];
        }
    };

    f32x16 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = f32x16{};

    const int nk = (K + kBK - 1) / kBK;
    gload(0);
    lstore(0);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
        const int cur = kt & 1;
        if (kt + 1 < nk) gload((kt + 1) * kBK);
#pragma unroll
        for (int s = 0; s < kBK / 16; ++s) {
            const int c = s * 2 + (lane >> 5);
            bf16x8 af[TM], bfg[TN];
#pragma unroll
            for (int i = 0; i < TM; ++i) {
                const int row = wm * WTM + i * 32 + (lane & 31);
                af[i] = *(const bf16x8*)&As[cur][row * kBK + swz(row, c) * 8];
            }
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                const int row = wn * WTN + j * 32 + (lane & 31);
                bfg[j] = *(const bf16x8*)&Bs[cur][row * kBK + swz(row, c) * 8];
            }
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bfg[j], af[i], acc[i][j], 0, 0, 0);
        }
        if (kt + 1 < nk) lstore(cur ^ 1);
        __syncthreads();
    }

    // Operands were swapped (B rows first), so lane l holds output row (l & 31) and
    // four consecutive output columns per group of four accumulators.
#pragma unroll
    for (int i = 0; i < TM; ++i) {
        const int m = m0 + wm * WTM + i * 32 + (lane & 31);
        if (m >= M) continue;
#pragma unroll
        for (int j = 0; j < TN; ++j) {
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int n = n0 + wn * WTN + j * 32 + 8 * g + 4 * (lane >> 5);
                const float v0 = acc[i][j][4 * g], v1 = acc[i][j][4 * g + 1];
                const float v2 = acc[i][j][4 * g + 2], v3 = acc[i][j][4 * g + 3];
                if constexpr (C_F32) {
                    float* p = (float*)Cp + (int64_t)m * ldc + n;
                    if (n + 3 < N) {
                        *(float4*)p = make_float4(v0, v1, v2, v3);
                    } else {
                        if (n < N) p[0] = v0;
                        if (n + 1 < N) p[1] = v1;
                        if (n + 2 < N) p[2] = v2;
                    }
                } else {
                    bf16* p = (bf16*)Cp + (int64_t)m * ldc + n;
                    if (n + 3 < N) {
                        bf16x4 o;
                        o[0] = (bf16)v0; o[1] = (bf16)v1; o[2] = (bf16)v2; o[3] = (bf16)v3;
                        *(bf16x4*)p = o;
                    } else {
                        if (n < N) p[0] = (bf16)v0;
                        if (n + 1 < N) p[1] = (bf16)v1;
                        if (n + 2 < N) p[2] = (bf16)v2;
                    }
                }
            }
        }
    }
}

// f(integral_constant<int, i>) for i = 0 .. N-1, unrolled at compile time
template <typename F, int... I>
__device__ __forceinline__ void static_for_seq(F&& f, std::integer_sequence<int, I...>) {
    (f(std::integral_constant<int, I>{}), ...);
}
template <int N, typename F> __device__ __forceinline__ void static_for(F&& f) {
    static_for_seq(f, std::make_integer_sequence<int, N>{});
}

// bf16 operands, K a multiple of BK: tiles move global -> LDS on the DMA path
// (buffer_load_dwordx4 ... lds: each lane writes 16 bytes at its lane slot of a 1 KB LDS
// block), so there are no staging registers and no ds_write instructions. A lane picks
// the global chunk that belongs at its slot under the XOR swizzle. The LDS holds a ring
// of NS stages, NS-1 tiles ahead of the one being multiplied (two schedules, below). The
// DMA is issued from inline assembly
// (M0 = LDS destination) and its completion is awaited by explicit vmcnt waits, so the
// compiler does not serialise the prefetch behind each tile's LDS reads. Rows past M
// or N are clamped to a valid row (their results are never stored). Fragments of
// k-substep s+1 are read from LDS while the MFMAs of substep s run.
// chunk permutation of an LDS row: 16 lanes reading one chunk column of 16 consecutive
// rows hit distinct 16-byte bank groups (128-byte rows: key (r>>1)&7; 64-byte: (r>>2)&3)
template <int BK> __device__ __forceinline__ int swz_k(int row, int chunk) {
    if constexpr (BK == 64) return chunk ^ ((row >> 1) & 7);
    else return chunk ^ ((row >> 2) & 3);
}

// WM x WN waves; with 8 waves two share each SIMD, so one wave's barrier and LDS waits
// are covered by the other's MFMAs. SPLIT: workgroup (tile, blockIdx.y) multiplies the
// K-slice [blockIdx.y * K, (blockIdx.y + 1) * K) (K is the slice length) and stores its
// fp32 partial tile at part[blockIdx.y][M][N]; a reduce kernel adds the slices.
// F32: the operands are float32 rows passed as bf16 rows of twice the length (K, lda and
// ldb in bf16 units); the DMA and the LDS layout only move bytes, and each 16-byte fragment
// (4 floats along k) feeds four v_mfma_f32_32x32x2_f32 instead of one bf16 MFMA.
// MB16: 16x16 MFMA blocks. FINE: the second, fully ordered schedule of the k loop. SB (with
// FINE): one set of weight fragments, each reloaded right after its last MFMA of a substep
// (the MFMAs run weight block by weight block), which frees registers for wider tiles.
template <int ROLE, int BM, int BN, int BK, int NS, int WM, int WN, bool C_F32, bool SPLIT = false, bool F32 = false,
          bool MB16 = false, bool FINE = false, bool SB = false>
__global__ __launch_bounds__(64 * WM * WN) void gemm_bf16_dma(int M, int N, int K, const bf16* __restrict__ A,
                                                              int64_t lda, const bf16* __restrict__ B, int64_t ldb,
                                                              void* __restrict__ Cp, int64_t ldc, int tiles_m,
                                                              int tiles_n, float* __restrict__ part) {
    constexpr int NW = WM * WN;
    constexpr int WTM = BM / WM, WTN = BN / WN;
    // MFMA blocks: 32x32 (bf16 32x32x16 or fp32 32x32x2), or 16x16 (MB16: bf16 16x16x32 or
    // fp32 16x16x4)
    constexpr int BLK = MB16 ? 16 : 32;
    constexpr int TM = WTM / BLK, TN = WTN / BLK;
    static_assert(TM * BLK == WTM && TN * BLK == WTN, "whole MFMA blocks per wave");
    using AccT = typename std::conditional<MB16, f32x4, f32x16>::type;
    constexpr int QG = MB16 ? 1 : 4;        // float4 groups of an accumulator
    constexpr int CPR = BK / 8;             // 16-byte chunks per row
    constexpr int RPB = 64 / CPR;           // rows per 1 KB DMA block
    // DMA blocks of one stage: BM / RPB activation blocks, then BN / RPB weight blocks. When
    // they split evenly, wave w takes AG consecutive activation and BG weight blocks;
    // otherwise (a 2-deep ring only, whose waits are for all of a wave's loads) block b goes to
    // wave b % NW, so waves take QM or QM - 1 blocks
    constexpr bool EVEN = BM % (RPB * NW) == 0 && BN % (RPB * NW) == 0;
    constexpr int TBA = BM / RPB, TBT = (BM + BN) / RPB, QM = (TBT + NW - 1) / NW;
    constexpr int AG = EVEN ? BM / RPB / NW : 0, BG = EVEN ? BN / RPB / NW : 0;  // DMA blocks per wave per stage
    constexpr int OPS = EVEN ? AG + BG : QM;
    constexpr int SUB = MB16 ? BK / 32 : BK / 16;  // MFMA k-substeps per stage (2 or 4 chunks of a row each)
    static_assert(NS >= 2 && BM % RPB == 0 && BN % RPB == 0, "tile");
    static_assert(EVEN ? (AG >= 1 && BG >= 1) : NS == 2, "uneven DMA blocks need the 2-deep ring");
    static_assert(SUB % 2 == 0, "fragment sets alternate within a tile");
    // one LDS block: the operand ring, reused after the k loop to stage the output tile
    constexpr int RING = NS * (BM + BN) * BK * 2;
    using OT = typename std::conditional<C_F32 || SPLIT, float, bf16>::type;
    // stage the output tile (or a K-slice's fp32 partial tile) through LDS, in one or two
    // passes of whole wave rows: whole-line stores instead of the MFMA layout's 16-byte
    // pieces spread over 32 rows
    constexpr int PASSES = (BM * BN * (int)sizeof(OT) + RING - 1) / RING;
    constexpr int RB = BM / PASSES;  // tile rows per pass
    constexpr bool STAGE = (BN * (int)sizeof(OT)) % 128 == 0 && PASSES <= 2 && BM % PASSES == 0 &&
                           RB % (BM / WM) == 0;
    __shared__ __attribute__((aligned(1024))) char smem[RING];
    bf16 (*As)[BM * BK] = reinterpret_cast<bf16 (*)[BM * BK]>(smem);
    bf16 (*Bs)[BN * BK] = reinterpret_cast<bf16 (*)[BN * BK]>(smem + NS * BM * BK * 2);

    int tm, tn;
    tile_of(tiles_m, tiles_n, tm, tn);
    const int m0 = tm * BM, n0 = tn * BN;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave / WN, wn = wave % WN;
    if constexpr (SPLIT) {
        A += (int64_t)blockIdx.y * K;
        B += (int64_t)blockIdx.y * K;
    }

    const int lr = lane / CPR, lp = lane % CPR;
    // the tile's row panels as buffer resources; a lane's chunk is a fixed byte offset in
    // them and the k advance goes in the scalar offset
    const __amdgpu_buffer_rsrc_t ra = buffer_rsrc(A + (int64_t)m0 * lda, (uint32_t)((int64_t)min(BM, M - m0) * lda * 2));
    const __amdgpu_buffer_rsrc_t rbr = buffer_rsrc(B + (int64_t)n0 * ldb, (uint32_t)((int64_t)min(BN, N - n0) * ldb * 2));
    auto a_off = [&](int r) { return (uint32_t)(((int64_t)(min(m0 + r, M - 1) - m0) * lda + swz_k<BK>(r, lp) * 8) * 2); };
    auto b_off = [&](int r) { return (uint32_t)(((int64_t)(min(n0 + r, N - 1) - n0) * ldb + swz_k<BK>(r, lp) * 8) * 2); };
    const uint32_t a_lds = (uint32_t)(uintptr_t)(lds_ptr_t)&As[0][0];
    const uint32_t b_lds = (uint32_t)(uintptr_t)(lds_ptr_t)&Bs[0][0];
    constexpr int NA = EVEN ? AG : QM, NB = EVEN ? BG : 1;
    uint32_t aoff[NA], boff[NB];
    const int wu = __builtin_amdgcn_readfirstlane(wave);  // wave-uniform, for the block choice
    if constexpr (EVEN) {
#pragma unroll
        for (int q = 0; q < AG; ++q) aoff[q] = a_off((wave * AG + q) * RPB + lr);
#pragma unroll
        for (int q = 0; q < BG; ++q) boff[q] = b_off((wave * BG + q) * RPB + lr);
    } else {
#pragma unroll
        for (int q = 0; q < QM; ++q) {
            const int b = wu + NW * q;
            aoff[q] = b < TBA ? a_off(b * RPB + lr) : b_off((b - TBA) * RPB + lr);
        }
    }
    auto dma = [&](int kt, int stage) {
        const int k0 = kt * BK;
        if constexpr (EVEN) {
#pragma unroll
            for (int q = 0; q < AG; ++q)
                dma16(ra, aoff[q], (uint32_t)k0 * 2, __builtin_amdgcn_readfirstlane(a_lds + (uint32_t)((stage * BM + (wave * AG + q) * RPB) * BK * 2)));
#pragma unroll
            for (int q = 0; q < BG; ++q)
                dma16(rbr, boff[q], (uint32_t)k0 * 2, __builtin_amdgcn_readfirstlane(b_lds + (uint32_t)((stage * BN + (wave * BG + q) * RPB) * BK * 2)));
        } else {
#pragma unroll
            for (int q = 0; q < QM; ++q) {
                const int b = wu + NW * q;
                if (b < TBA)
                    dma16(ra, aoff[q], (uint32_t)k0 * 2, a_lds + (uint32_t)((stage * BM + b * RPB) * BK * 2));
                else if (b < TBT)
                    dma16(rbr, aoff[q], (uint32_t)k0 * 2, b_lds + (uint32_t)((stage * BN + (b - TBA) * RPB) * BK * 2));
            }
        }
    };

    AccT acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = AccT{};
    // a lane's fragment rows are wm * WTM + i * BLK + lane % BLK: the block offsets are
    // multiples of 16 rows, which leave the swizzle key (row bits 1-3, or 2-3 for 32-wide
    // stages) unchanged, so block i is a constant offset from block 0 and every fragment
    // address is one per-lane base plus an immediate
    static_assert(WTM % 16 == 0 && WTN % 16 == 0 && BLK % 16 == 0, "swizzle key per lane");
    const int arow0 = wm * WTM + (lane & (BLK - 1)), brow0 = wn * WTN + (lane & (BLK - 1));
    // lane l's output columns of float4 group g of a block (its row is l % BLK): the MFMA
    // layouts with the weight fragment as the first operand
    auto ocol = [&](int g) { return MB16 ? 4 * (lane >> 4) : 8 * g + 4 * (lane >> 5); };

    const int nk = K / BK;
    bf16x8 fa[2][TM], fb[2][TN];
    auto frag = [&](int stage, int s, int set) {
        const bf16* as = As[stage];
        const bf16* bs = Bs[stage];
        const int c = MB16 ? s * 4 + (lane >> 4) : s * 2 + (lane >> 5);
#pragma unroll
        for (int i = 0; i < TM; ++i) fa[set][i] = *(const bf16x8*)&as[(arow0 + i * BLK) * BK + swz_k<BK>(arow0, c) * 8];
#pragma unroll
        for (int j = 0; j < TN; ++j) fb[set][j] = *(const bf16x8*)&bs[(brow0 + j * BLK) * BK + swz_k<BK>(brow0, c) * 8];
    };
    auto mfma = [&](int set) {
        if constexpr (MB16 && !F32) {
            // bf16 on 16x16 blocks: lane group g = l / 16 takes chunk 4s + g, the 8 values of
            // k = 32s + 8g .. 32s + 8g + 7 that v_mfma_f32_16x16x32_bf16 expects of it
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fb[set][j], fa[set][i], acc[i][j], 0, 0, 0);
        } else if constexpr (MB16) {
            // float32 operands on 16x16 blocks: lane group g = l / 16 takes chunk 4s + g, so
            // MFMA u sums k = 16s + 4g + u over the four groups
#pragma unroll
            for (int u = 0; u < 4; ++u)
#pragma unroll
                for (int i = 0; i < TM; ++i)
#pragma unroll
                    for (int j = 0; j < TN; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(__builtin_bit_cast(f32x4, fb[set][j])[u],
                                                                         __builtin_bit_cast(f32x4, fa[set][i])[u],
                                                                         acc[i][j], 0, 0, 0);
        } else if constexpr (F32) {
            // float32 operands: a 16-byte chunk holds 4 floats along k; lanes 0-31 take chunk
            // 2s, lanes 32-63 chunk 2s + 1, so MFMA u sums k = 8s + u and 8s + 4 + u
#pragma unroll
            for (int u = 0; u < 4; ++u)
#pragma unroll
                for (int i = 0; i < TM; ++i)
#pragma unroll
                    for (int j = 0; j < TN; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(__builtin_bit_cast(f32x4, fb[set][j])[u],
                                                                         __builtin_bit_cast(f32x4, fa[set][i])[u],
                                                                         acc[i][j], 0, 0, 0);
        } else {
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fb[set][j], fa[set][i], acc[i][j], 0, 0, 0);
        }
    };
    // one MFMA per fragment read, then the remaining MFMAs of the substep
    constexpr int NMF = TM * TN * (F32 ? 4 : 1);
    auto interleave = [&]() {
#pragma unroll
        for (int q = 0; q < TM + TN; ++q) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        }
        if (NMF > TM + TN) __builtin_amdgcn_sched_group_barrier(0x008, NMF - (TM + TN), 0);
    };

    if constexpr (!FINE) {
        // First schedule: the DMA of tile kt+NS-1 goes out at the top of tile kt, all at once.
#pragma unroll
        for (int st = 0; st < NS - 1; ++st)
            if (st < nk) dma(st, st);
        // tile 0 complete: NS-2 newer tiles may stay in flight, unless K has fewer tiles than that
        if (nk >= NS - 1) wait_vm<(NS - 2) * OPS>();
        else wait_vm<0>();
        __syncthreads();
        frag(0, 0, 0);
        for (int kt = 0; kt < nk; ++kt) {
            const int cur = kt % NS;
            if (kt + NS - 1 < nk) dma(kt + NS - 1, (kt + NS - 1) % NS);
            // substeps 0 .. SUB-2, each reading the fragments of the next
#pragma unroll
            for (int s = 0; s + 1 < SUB; ++s) {
                frag(cur, s + 1, (s + 1) & 1);
                mfma(s & 1);
                interleave();
            }
            // Tile kt+1 must be complete in LDS (this wave's DMA, then all waves'), and this
            // wave's reads of stage cur must be done before anyone refills it. The barrier
            // sits before the last substep so its MFMAs cover the first reads of tile kt+1.
            if (kt + 1 < nk) {
                const int newer = min(NS - 2, nk - 2 - kt);  // tiles newer than kt+1 in flight
                if (newer >= NS - 2) wait_vm<(NS - 2) * OPS>();
                else wait_vm<0>();  // tail: wait for everything
            }
            __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): fragments of the last substep are in
            __syncthreads();
            if (kt + 1 < nk) frag((kt + 1) % NS, 0, SUB & 1);
            mfma((SUB - 1) & 1);
            interleave();
        }
    } else {
    // Second schedule: every load, fragment read and MFMA in a fixed order. A stage is
    // refilled as soon as every wave has read its last fragments (at the barrier one substep
    // before the end of its tile), with the DMA blocks spread one every few MFMAs, so a wave
    // never waits behind a run of its own loads while the MFMA pipe idles.
    // One DMA block d of tile kt into stage `stage`, from resources rA / rB (the panels, or
    // empty resources: a load past the last tile then reads nothing and writes zeros into a
    // stage that is never read again, which keeps every wave's load count the same)
    auto dma_one = [&](int kt, int stage, auto D, __amdgpu_buffer_rsrc_t rA, __amdgpu_buffer_rsrc_t rB)
                       __attribute__((always_inline)) {
        constexpr int d = decltype(D)::value;
        const uint32_t k2 = (uint32_t)(kt * BK) * 2;
        if constexpr (EVEN) {
            if constexpr (d < AG)
                dma16(rA, aoff[d], k2, __builtin_amdgcn_readfirstlane(a_lds + (uint32_t)((stage * BM + (wave * AG + d) * RPB) * BK * 2)));
            else
                dma16(rB, boff[d - AG], k2, __builtin_amdgcn_readfirstlane(b_lds + (uint32_t)((stage * BN + (wave * BG + d - AG) * RPB) * BK * 2)));
        } else {
            const int b = wu + NW * d;
            if (b < TBA)
                dma16(rA, aoff[d], k2, a_lds + (uint32_t)((stage * BM + b * RPB) * BK * 2));
            else if (b < TBT)
                dma16(rB, aoff[d], k2, b_lds + (uint32_t)((stage * BN + (b - TBA) * RPB) * BK * 2));
        }
    };
    const __amdgpu_buffer_rsrc_t ra_none = buffer_rsrc(A, 0), rb_none = buffer_rsrc(B, 0);
    // every DMA block of tile kt into stage `stage` (none past the last tile)
    auto dma_all = [&](int kt, int stage) __attribute__((always_inline)) {
        const bool live = kt < nk;
        static_for<OPS>([&](auto D) __attribute__((always_inline)) {
            dma_one(kt, stage, D, live ? ra : ra_none, live ? rbr : rb_none);
        });
    };
    // fragment f (activation blocks, then weight blocks) of substep s of stage `stage`
    auto frag_one = [&](int stage, int s, auto SET, auto F) __attribute__((always_inline)) {
        constexpr int set = decltype(SET)::value, f = decltype(F)::value;
        const int c = MB16 ? s * 4 + (lane >> 4) : s * 2 + (lane >> 5);
        if constexpr (f < TM) fa[set][f] = *(const bf16x8*)&As[stage][(arow0 + f * BLK) * BK + swz_k<BK>(arow0, c) * 8];
        else fb[SB ? 0 : set][f - TM] = *(const bf16x8*)&Bs[stage][(brow0 + (f - TM) * BLK) * BK + swz_k<BK>(brow0, c) * 8];
    };
    // MFMA q of a substep (block row by block row; with SB block column by block column)
    static_assert(!F32, "the second schedule is for bf16 operands (the float32 tiles keep the first)");
    auto mfma_one = [&](auto SET, auto Q) __attribute__((always_inline)) {
        constexpr int set = decltype(SET)::value, q = decltype(Q)::value;
        constexpr int i = SB ? q % TM : q / TN, j = SB ? q / TM : q % TN, sb = SB ? 0 : set;
        if constexpr (MB16)
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fb[sb][j], fa[set][i], acc[i][j], 0, 0, 0);
        else
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fb[sb][j], fa[set][i], acc[i][j], 0, 0, 0);
    };
    // one substep: the NMF MFMAs of fragment set SET, with the reads of the other set
    // (substep rsub of stage rs) and, with DMA, the OPS refill blocks of tile dkt into stage
    // dst spread evenly between them; the order is pinned, so no wave issues a run of loads
    // while its MFMAs wait
    auto substep = [&](auto DMA, auto SET, int rs, int rsub, int dkt, int dst) __attribute__((always_inline)) {
        constexpr int set = decltype(SET)::value;
        const bool live = dkt < nk;
        const __amdgpu_buffer_rsrc_t rA = live ? ra : ra_none, rB = live ? rbr : rb_none;
        static_for<NMF>([&](auto Q) __attribute__((always_inline)) {
            constexpr int q = decltype(Q)::value;
            if constexpr (decltype(DMA)::value)
                static_for<OPS>([&](auto D) __attribute__((always_inline)) {
                    if constexpr (decltype(D)::value * NMF / OPS == q) dma_one(dkt, dst, D, rA, rB);
                });
            // the next set's reads go out first, one per MFMA, so they land early (with SB the
            // weight fragments only after their last MFMA here)
            static_for<SB ? TM : TM + TN>([&](auto F) __attribute__((always_inline)) {
                if constexpr ((decltype(F)::value < NMF ? decltype(F)::value : NMF - 1) == q)
                    frag_one(rs, rsub, std::integral_constant<int, set ^ 1>{}, F);
            });
            mfma_one(SET, Q);
            if constexpr (SB && q % TM == TM - 1)
                frag_one(rs, rsub, std::integral_constant<int, set ^ 1>{}, std::integral_constant<int, TM + q / TM>{});
            __builtin_amdgcn_sched_barrier(0);
        });
    };
    // Every wave issues OPS loads per tile for NS tiles ahead, tiles past the last included
    // (as loads of nothing), so every wait below is the same count.
    static_for<NS - 1>([&](auto ST) __attribute__((always_inline)) { dma_all(ST, ST); });
    wait_vm<(NS - 2) * OPS>();  // tile 0 complete
    dma_all(NS - 1, NS - 1);    // the last stage of the ring is free from the start
    __syncthreads();
    frag(0, 0, 0);
    for (int kt = 0; kt < nk; ++kt) {
        const int cur = kt % NS;
        // substeps 0 .. SUB-2, each reading the fragments of the next
        static_for<SUB - 1>([&](auto S) __attribute__((always_inline)) {
            constexpr int s = decltype(S)::value;
            substep(std::false_type{}, std::integral_constant<int, s & 1>{}, cur, s + 1, 0, 0);
        });
        // Tile kt+1 must be complete in LDS (this wave's DMA, then all waves'), and every
        // wave's reads of stage cur must be done before it is refilled. The barrier sits
        // before the last substep, so its MFMAs cover the first reads of tile kt+1, and the
        // refill of stage cur with tile kt+NS goes out between them: each tile's DMA has a
        // whole tile of MFMAs, from one barrier to the next, to land. (After the last tile
        // the reads of stage (kt+1) % NS fetch values that are never used.)
        wait_vm<(NS - 2) * OPS>();
        __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): fragments of the last substep are in
        __syncthreads();
        substep(std::true_type{}, std::integral_constant<int, (SUB - 1) & 1>{}, (kt + 1) % NS, 0, kt + NS, cur);
    }
    wait_vm<0>();  // the loads of nothing past the last tile write the ring too
    }

    if constexpr (STAGE) {
        // tile row r is stored as 16-byte chunks, chunk c at position c ^ (r & 7)
        constexpr int E16 = 16 / (int)sizeof(OT);   // elements per chunk
        constexpr int CPR_O = BN / E16;             // chunks per tile row
        OT* st = reinterpret_cast<OT*>(smem);
        // a K-slice's fp32 partial goes to part[blockIdx.y] (row stride N), the output to C
        OT* const out = SPLIT ? reinterpret_cast<OT*>(part + (int64_t)blockIdx.y * M * N) : (OT*)Cp;
        const int64_t ldo = SPLIT ? (int64_t)N : ldc;
        const bool vec = ((uintptr_t)out & 15) == 0 && (ldo * (int64_t)sizeof(OT)) % 16 == 0;
#pragma unroll
        for (int pass = 0; pass < PASSES; ++pass) {
            __syncthreads();  // every wave is done with the ring (then with the previous pass)
            if (wm * WTM >= pass * RB && wm * WTM < (pass + 1) * RB) {
#pragma unroll
                for (int i = 0; i < TM; ++i) {
                    const int r = wm * WTM - pass * RB + i * BLK + (lane & (BLK - 1));
#pragma unroll
                    for (int j = 0; j < TN; ++j)
#pragma unroll
                        for (int g = 0; g < QG; ++g) {
                            const int col = wn * WTN + j * BLK + ocol(g);
                            OT* q = st + r * BN + (((col / E16) ^ (r & 7)) * E16) + col % E16;
                            const float v0 = acc[i][j][4 * g], v1 = acc[i][j][4 * g + 1];
                            const float v2 = acc[i][j][4 * g + 2], v3 = acc[i][j][4 * g + 3];
                            if constexpr (sizeof(OT) == 4) {
                                *(float4*)q = make_float4(v0, v1, v2, v3);
                            } else {
                                bf16x4 o;
                                o[0] = (bf16)v0; o[1] = (bf16)v1; o[2] = (bf16)v2; o[3] = (bf16)v3;
                                *(bf16x4*)q = o;
                            }
                        }
                }
            }
            __syncthreads();
            for (int c = tid; c < RB * CPR_O; c += 64 * NW) {
                const int r = c / CPR_O, cc = c % CPR_O;
                const int m = m0 + pass * RB + r, n = n0 + cc * E16;
                if (m >= M || n >= N) continue;
                const OT* q = st + r * BN + ((cc ^ (r & 7)) * E16);
                OT* p = out + (int64_t)m * ldo + n;
                if (vec && n + E16 <= N) {
                    *(u32x4*)p = *(const u32x4*)q;
                } else {
                    for (int e = 0; e < E16 && n + e < N; ++e) p[e] = q[e];
                }
            }
        }
        return;
    }
#pragma unroll
    for (int i = 0; i < TM; ++i) {
        const int m = m0 + wm * WTM + i * BLK + (lane & (BLK - 1));
        if (m >= M) continue;
#pragma unroll
        for (int j = 0; j < TN; ++j) {
#pragma unroll
            for (int g = 0; g < QG; ++g) {
                const int n = n0 + wn * WTN + j * BLK + ocol(g);
                const float v0 = acc[i][j][4 * g], v1 = acc[i][j][4 * g + 1];
                const float v2 = acc[i][j][4 * g + 2], v3 = acc[i][j][4 * g + 3];
                if constexpr (SPLIT) {
                    float* p = part + ((int64_t)blockIdx.y * M + m) * N + n;
                    if (n + 3 < N && (N & 3) == 0) {
                        *(float4*)p = make_float4(v0, v1, v2, v3);
                    } else {
                        if (n < N) p[0] = v0;
                        if (n + 1 < N) p[1] = v1;
                        if (n + 2 < N) p[2] = v2;
                        if (n + 3 < N) p[3] = v3;
                    }
                } else if constexpr (C_F32) {
                    float* p = (float*)Cp + (int64_t)m * ldc + n;
                    if (n + 3 < N) {
                        *(float4*)p = make_float4(v0, v1, v2, v3);
                    } else {
                        if (n < N) p[0] = v0;
                        if (n + 1 < N) p[1] = v1;
                        if (n + 2 < N) p[2] = v2;
                    }
                } else {
                    bf16* p = (bf16*)Cp + (int64_t)m * ldc + n;
                    if (n + 3 < N) {
                        bf16x4 o;
                        o[0] = (bf16)v0; o[1] = (bf16)v1; o[2] = (bf16)v2; o[3] = (bf16)v3;
                        *(bf16x4*)p = o;
                    } else {
                        if (n < N) p[0] = (bf16)v0;
                        if (n + 1 < N) p[1] = (bf16)v1;
                        if (n + 2 < N) p[2] = (bf16)v2;
                    }
                }
            }
        }
    }
}

// C[m][n] = sum over the slices, in slice order, of part[slice][m][n]; 4 outputs per thread
template <bool C_F32>
__global__ __launch_bounds__(256) void splitk_reduce_kernel(const float* __restrict__ part, int splits, int M, int N,
                                                            void* __restrict__ Cp, int64_t ldc) {
    const int n4 = (N + 3) / 4;
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= (int64_t)M * n4) return;
    const int m = (int)(i / n4), n = (int)(i % n4) * 4;
    const int64_t slice = (int64_t)M * N;
    const float* p = part + (int64_t)m * N + n;
    float v[4] = {0.0f, 0.0f, 0.0f, 0.0f};
    const bool full = n + 3 < N && (N & 3) == 0;
    for (int sp = 0; sp < splits; ++sp, p += slice) {
        if (full) {
            const float4 q = *(const float4*)p;
            v[0] += q.x; v[1] += q.y; v[2] += q.z; v[3] += q.w;
        } else {
#pragma unroll
            for (int e = 0; e < 4; ++e)
                if (n + e < N) v[e] += p[e];
        }
    }
    if constexpr (C_F32) {
        float* c = (float*)Cp + (int64_t)m * ldc + n;
#pragma unroll
        for (int e = 0; e < 4; ++e)
            if (n + e < N) c[e] = v[e];
    } else {
        bf16* c = (bf16*)Cp + (int64_t)m * ldc + n;
#pragma unroll
        for (int e = 0; e < 4; ++e)
            if (n + e < N) c[e] = (bf16)v[e];
    }
}

template <int ROLE, int BM, int BN, int BK, int NS, int WM, int WN, bool CF, bool MB16 = false, bool FINE = false,
          bool SB = false>
hipError_t run_dma(int64_t M, int64_t N, int64_t K, const void* A, int64_t lda, const void* B, int64_t ldb, void* C,
                   int64_t ldc, hipStream_t s, int splits = 1, float* part = nullptr) {
    const int tm = (int)((M + BM - 1) / BM), tn = (int)((N + BN - 1) / BN);
    if (splits <= 1) {
        SSM_LAUNCH((gemm_bf16_dma<ROLE, BM, BN, BK, NS, WM, WN, CF, false, false, MB16, FINE, SB>), dim3(tm * tn), dim3(64 * WM * WN), 0, s,
                   (int)M, (int)N, (int)K, (const bf16*)A, lda, (const bf16*)B, ldb, C, ldc, tm, tn, nullptr);
        return hipGetLastError();
    }
    SSM_LAUNCH((gemm_bf16_dma<ROLE, BM, BN, BK, NS, WM, WN, CF, true, false, MB16, FINE, SB>), dim3(tm * tn, splits), dim3(64 * WM * WN), 0,
               s, (int)M, (int)N, (int)(K / splits), (const bf16*)A, lda, (const bf16*)B, ldb, C, ldc, tm, tn, part);
    if (const hipError_t e = hipGetLastError(); e != hipSuccess) return e;
    KernelTimer kt("gemm.splitk_reduce", s);
    const int64_t n = M * ((N + 3) / 4);
    SSM_LAUNCH((splitk_reduce_kernel<CF>), dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, (const float*)part,
               splits, (int)M, (int)N, C, ldc);
    return hipGetLastError();
}

// float32 operands on the DMA tiles: the rows are moved as bytes, so the kernel sees them as
// bf16 rows of twice the length (K, lda, ldb doubled); only the MFMAs read them as floats
template <int ROLE, int BM, int BN, int NS, int WM, int WN, bool MB16 = false>
hipError_t run_dma_f32(int64_t M, int64_t N, int64_t K, const float* A, int64_t lda, const float* B, int64_t ldb,
                       float* C, int64_t ldc, hipStream_t s, int splits = 1, float* part = nullptr) {
    const int tm = (int)((M + BM - 1) / BM), tn = (int)((N + BN - 1) / BN);
    if (splits <= 1) {
        SSM_LAUNCH((gemm_bf16_dma<ROLE, BM, BN, 64, NS, WM, WN, true, false, true, MB16>), dim3(tm * tn), dim3(64 * WM * WN),
                   0, s, (int)M, (int)N, (int)(2 * K), (const bf16*)A, 2 * lda, (const bf16*)B, 2 * ldb, C, ldc, tm,
                   tn, nullptr);
        return hipGetLastError();
    }
    SSM_LAUNCH((gemm_bf16_dma<ROLE, BM, BN, 64, NS, WM, WN, true, true, true, MB16>), dim3(tm * tn, splits),
               dim3(64 * WM * WN), 0, s, (int)M, (int)N, (int)(2 * K / splits), (const bf16*)A, 2 * lda,
               (const bf16*)B, 2 * ldb, C, ldc, tm, tn, part);
    if (const hipError_t e = hipGetLastError(); e != hipSuccess) return e;
    KernelTimer kt("gemm.splitk_reduce", s);
    const int64_t n4 = M * ((N + 3) / 4);
    SSM_LAUNCH((splitk_reduce_kernel<true>), dim3((unsigned)((n4 + 255) / 256)), dim3(256), 0, s, (const float*)part,
               splits, (int)M, (int)N, C, ldc);
    return hipGetLastError();
}

// Tile shape by a wave-quantisation cost model: whole rounds of 256 workgroups (one per
// CU) times tile area over the shape's measured efficiency (256x256 does the most MFMA
// work per LDS byte; 128x128 gives more workgroups when the grid is small). 256x320 (4x2
// waves of 64x160) takes an output whose 256-wide tiles leave the last round part-empty
// but whose N is a multiple of 320: out_proj of the 2.8B half shard (16384 x 2560) runs
// 512 of them in 2 rounds instead of 640 256x256 tiles in 3. All three run on 16x16 blocks
// with the second schedule (5-7% faster than 32x32 blocks with the first): 256x256 as 2x4
// waves of 128x64, 128x128 as 2x2 waves of 64x64 (two workgroups per CU), 256x320 as 4x2
// waves of 64x160 with one set of weight fragments (two sets do not fit in the registers).
enum DmaTiles { kTiles128 = 0, kTiles256 = 1, kTiles256x320 = 2 };
DmaTiles dma_tiles(int64_t M, int64_t N) {
    auto cost = [&](int bm, int bn, double eff) {
        const int64_t tiles = ((M + bm - 1) / bm) * ((N + bn - 1) / bn);
        return (double)((tiles + 255) / 256) * bm * bn / eff;
    };
    const double c256 = cost(256, 256, 1.0);
    if (c256 > cost(128, 128, 0.83)) return kTiles128;
    return (N % 320 == 0 && cost(256, 320, 1.0) < c256) ? kTiles256x320 : kTiles256;
}
bool dma_big_tiles(int64_t M, int64_t N) { return dma_tiles(M, N) != kTiles128; }

// Float32 tiles by the same kind of model: rounds of workgroups (one per CU; two for the 64 KB
// ring of 128x128) times the work a CU does per round over the tile's measured per-CU MFMA
// efficiency. On the hybrid shard's 2048-row chunks: 256x256 tiles (8 waves of 128x64) 0.91,
// 256x224 (8 waves of 32x224) 0.93, 128x224 (8 waves of 32x112 on 16x16 blocks) 0.91,
// 128x128 (8 waves of 64x32, two per CU) 0.89. The 224-wide tiles exist for outputs whose
// 256-wide tiles leave part of a round empty: in_proj (2048 x 7168) takes 256 tiles of 256x224
// where 256x256 gave 224 (840 -> 720 us), out_proj (2048 x 3584) 256 tiles of 128x224 where
// 128x128 gave 448 over two slots per CU (430 -> 368 us; 4 waves of 32x224, one per SIMD,
// took 393 us; 64x112 wave tiles on 16x16 blocks for 256x224 spill).
enum F32Tiles { kF32Tiles128 = 0, kF32Tiles256 = 1, kF32Tiles256x224 = 2, kF32Tiles128x224 = 3, kF32Tiles64 = 4 };
F32Tiles f32_tiles(int64_t M, int64_t N) {
    auto cost = [&](int bm, int bn, int per_cu, double eff) {
        const int64_t tiles = ((M + bm - 1) / bm) * ((N + bn - 1) / bn), slots = 256 * per_cu;
        return (double)((tiles + slots - 1) / slots) * per_cu * bm * bn / eff;
    };
    F32Tiles best = kF32Tiles128;
    double c = cost(128, 128, 2, 0.89);
    const double c256 = cost(256, 256, 1, 0.91), c224 = cost(256, 224, 1, 0.93), c128x224 = cost(128, 224, 1, 0.91);
    if (c256 < c) { c = c256; best = kF32Tiles256; }
    if (c224 < c) { c = c224; best = kF32Tiles256x224; }
    if (c128x224 < c) { c = c128x224; best = kF32Tiles128x224; }
    return best;
}

// Decode batches above the few-row kernels (65..512 rows) with bf16 output: the streamed
// tile kernel of the decode projections (launch_gemm_skinny) when its tiles give at least
// 128 workgroups, without K-slices
bool decode_tiles(int64_t M, int64_t N, int64_t K) {
    return K % 64 == 0 && M > 64 && M <= 512 && ((M + 31) / 32) * ((N + 31) / 32) >= 128;
}
// x_proj of a decode batch (up to 512 rows, at most 256 columns): 16-row tiles of the
// few-row kernel, which spread over more workgroups than 64-row tiles and need no K-slices
bool xproj_decode_skinny(int64_t M, int64_t N) { return M <= 512 && N <= 256; }

// Split-K for outputs of fewer tiles than CUs: K is cut into equal slices of whole
// 64-wide k-tiles (at least two per slice) so that up to ~384 workgroups run; the slices'
// fp32 partials are added by a reduce kernel in slice order (deterministic).
int splitk_slices(int64_t tiles, int64_t K) {
    if (K % 64 != 0 || tiles >= 256) return 1;
    const int64_t nk = K / 64, cap = std::max<int64_t>(1, 384 / tiles);
    int best = 1;
    for (int64_t d = 2; d <= cap && d <= nk / 2; ++d)
        if (nk % d == 0) best = (int)d;
    return best;
}

int fit_slices(int sp, int64_t M, int64_t N, size_t scratch_bytes) {
    return (sp > 1 && (size_t)sp * M * N * 4 <= scratch_bytes) ? sp : 1;
}

template <int ROLE, bool CF>
hipError_t dispatch_dma(int64_t M, int64_t N, int64_t K, const void* A, int64_t lda, const void* B, int64_t ldb,
                        void* C, int64_t ldc, hipStream_t s, float* scratch, size_t scratch_bytes) {
    if (K % 64 == 0) {
        const DmaTiles t = dma_tiles(M, N);
        if (t == kTiles256x320)
            return run_dma<ROLE, 256, 320, 64, 2, 4, 2, CF, true, true, true>(M, N, K, A, lda, B, ldb, C, ldc, s);
        if (t == kTiles256) return run_dma<ROLE, 256, 256, 64, 2, 2, 4, CF, true, true>(M, N, K, A, lda, B, ldb, C, ldc, s);
    }
    if (K % 64 == 0) {
        const int sp = fit_slices(splitk_slices(((M + 127) / 128) * ((N + 127) / 128), K), M, N, scratch_bytes);
        return run_dma<ROLE, 128, 128, 64, 2, 2, 2, CF, true, true>(M, N, K, A, lda, B, ldb, C, ldc, s, sp, scratch);
    }
    // K a multiple of 32 only (dt_proj: K = dt_rank): a 3-slot ring (48 KB) lets three
    // workgroups share a CU, which shortens the many short-lived tiles' latency rounds
    // (dt_proj of 16384 tokens, K = 160: 35 -> 30 us against a 4-slot ring)
    return run_dma<ROLE, 128, 128, 32, 3, 2, 2, CF>(M, N, K, A, lda, B, ldb, C, ldc, s);
}

// fp32 weights and at most 8 activation rows (a decode step of the fp32 configuration),
// where the time is the weight read: one weight row per wave, streamed in 1 KB runs (64
// lanes x 4 floats, whole cache lines) and multiplied by the activation rows (M x K floats,
// shared by every wave and served from cache); the lanes' sums meet by xor shuffles. K,
// the leading dimensions and the pointers are multiples of 4 floats (checked by the caller).
template <int ROLE>
__global__ __launch_bounds__(256) void gemv_f32_kernel(int M, int N, int K, const float* __restrict__ A,
                                                       int64_t lda, const float* __restrict__ B, int64_t ldb,
                                                       float* __restrict__ C, int64_t ldc) {
    constexpr int MR = 8;
    const int lane = threadIdx.x & 63;
    const int n = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (n >= N) return;
    const float* brow = B + (int64_t)n * ldb;
    float acc[MR];
#pragma unroll
    for (int m = 0; m < MR; ++m) acc[m] = 0.0f;
    // four 1 KB runs per iteration, so that their loads are in flight together
    for (int k0 = lane * 4; k0 < K; k0 += 1024) {
        float4 b[4];
#pragma unroll
        for (int j = 0; j < 4; ++j)
            b[j] = k0 + 256 * j < K ? *(const float4*)(brow + k0 + 256 * j) : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
        for (int m = 0; m < MR; ++m) {
            if (m < M) {
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    if (k0 + 256 * j < K) {
                        const float4 a = *(const float4*)(A + (int64_t)m * lda + k0 + 256 * j);
                        acc[m] += a.x * b[j].x + a.y * b[j].y + a.z * b[j].z + a.w * b[j].w;
                    }
                }
            }
        }
    }
    float mine = 0.0f;
#pragma unroll
    for (int m = 0; m < MR; ++m) {
        if (m < M) {
            float v = acc[m];
#pragma unroll
            for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off);
            if (lane == m) mine = v;
        }
    }
    if (lane < M) C[(int64_t)lane * ldc + n] = mine;
}

// fp32 operands on v_mfma_f32_16x16x4_f32: 64x64 tiles, k 16 per stage, four waves of 32x32.
constexpr int kFBK = 16;
constexpr int kFPad = kFBK + 1;

template <int ROLE>
__global__ __launch_bounds__(256) void gemm_f32_nt(int M, int N, int K, const float* __restrict__ A,
                                                   int64_t lda, const float* __restrict__ B, int64_t ldb,
                                                   float* __restrict__ C, int64_t ldc, int tiles_m, int tiles_n) {
    __shared__ float As[2][64 * kFPad];
    __shared__ float Bs[2][64 * kFPad];
    int tm, tn;
    tile_of(tiles_m, tiles_n, tm, tn);
    const int m0 = tm * 64, n0 = tn * 64;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int lrow = tid >> 2, lck = tid & 3;  // one float4 of A and of B per thread
    float4 ra, rb;
    auto gload = [&](int k0) {
        const int gk = k0 + lck * 4;
        const int gm = m0 + lrow, gn = n0 + lrow;
        ra = (gm < M && gk < K) ? *(const float4*)(A + (int64_t)gm * lda + gk) : make_float4(0, 0, 0, 0);
        rb = (gn < N && gk < K) ? *(const float4*)(B + (int64_t)gn * ldb + gk) : make_float4(0, 0, 0, 0);
    };
    auto lstore = [&](int buf) {
        float* a = &As[buf][lrow * kFPad + lck * 4];
        float* b = &Bs[buf][lrow * kFPad + lck * 4];
        a[0] = ra.x; a[1] = ra.y; a[2] = ra.z; a[3] = ra.w;
        b[0] = rb.x; b[1] = rb.y; b[2] = rb.z; b[3] = rb.w;
    };
    f32x4 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = f32x4{};
    const int nk = (K + kFBK - 1) / kFBK;
    gload(0);
    lstore(0);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
        const int cur = kt & 1;
        if (kt + 1 < nk) gload((kt + 1) * kFBK);
#pragma unroll
        for (int s = 0; s < kFBK / 4; ++s) {
            float af[2], bfv[2];
#pragma unroll
            for (int i = 0; i < 2; ++i) af[i] = As[cur][(wm * 32 + i * 16 + (lane & 15)) * kFPad + s * 4 + (lane >> 4)];
#pragma unroll
            for (int j = 0; j < 2; ++j) bfv[j] = Bs[cur][(wn * 32 + j * 16 + (lane & 15)) * kFPad + s * 4 + (lane >> 4)];
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(bfv[j], af[i], acc[i][j], 0, 0, 0);
        }
        if (kt + 1 < nk) lstore(cur ^ 1);
        __syncthreads();
    }
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const int m = m0 + wm * 32 + i * 16 + (lane & 15);
        if (m >= M) continue;
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int n = n0 + wn * 32 + j * 16 + 4 * (lane >> 4);
            float* p = C + (int64_t)m * ldc + n;
            if (n + 3 < N) {
                *(float4*)p = make_float4(acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]);
            } else {
#pragma unroll
                for (int v = 0; v < 4; ++v)
                    if (n + v < N) p[v] = acc[i][j][v];
            }
        }
    }
}

// float32 k stages: 32 floats, one 128-byte line of every operand row
constexpr int kF32BK = 32;

// K-slices for a float32 product with few 128x128 tiles: the most slices (dividing the
// 32-wide stages, at least 4 stages each) that keep the grid within about two workgroups
// per CU. 1 = unsplit.
int f32_slices(int64_t tiles, int64_t K) {
    if (K % kF32BK != 0 || tiles >= 256) return 1;
    const int64_t nk = K / kF32BK, cap = std::max<int64_t>(1, 512 / tiles);
    int best = 1;
    for (int64_t d = 2; d <= cap && d <= nk / 4; ++d)
        if (nk % d == 0) best = (int)d;
    return best;
}

template <int ROLE, int BM, int BN, int WM, int WN, bool AF, bool CF>
hipError_t run_bf16(int64_t M, int64_t N, int64_t K, const void* A, int64_t lda, const void* B, int64_t ldb,
                    void* C, int64_t ldc, hipStream_t s) {
    const int tm = (int)((M + BM - 1) / BM), tn = (int)((N + BN - 1) / BN);
    SSM_LAUNCH((gemm_bf16_nt<ROLE, BM, BN, WM, WN, AF, CF>), dim3(tm * tn), dim3(256), 0, s, (int)M, (int)N,
                       (int)K, A, lda, (const bf16*)B, ldb, C, ldc, tm, tn);
    return hipGetLastError();
}

// o[m][k] = bf16(a[m][k]) (round to nearest even), 8 values per thread; K % 8 == 0
__global__ __launch_bounds__(256) void round_bf16_rows_kernel(const float* __restrict__ a, int64_t lda,
                                                              bf16* __restrict__ o, int64_t M, int K) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const int kg = K / 8;
    if (i >= M * kg) return;
    const int64_t m = i / kg;
    const int k = (int)(i % kg) * 8;
    const float* p = a + m * lda + k;
    *(bf16x8*)(o + m * K + k) = cvt8(*(const float4*)p, *(const float4*)(p + 4));
}

template <int ROLE, bool AF, bool CF>
hipError_t dispatch_bf16(int64_t M, int64_t N, int64_t K, const void* A, int64_t lda, const void* B, int64_t ldb,
                         void* C, int64_t ldc, hipStream_t s, float* scratch, size_t scratch_bytes) {
    // Tile by output size: large outputs use 256x256 (each wave 128x128, the most
    // MFMA work per LDS byte), mid-size ones 128x128 for more workgroups.
    // few rows: the weight read dominates; stream it with many narrow workgroups. fp32-A
    // dt_proj of a large decode batch (K = dt_rank) goes the same way: its staged 128x128
    // tiles would give only a few workgroups (20 for 256 sequences of a 1280-channel shard)
    if (M <= 64 || (ROLE == kGemmDtProj && AF && M <= 512 && K <= 512) ||
        (ROLE == kGemmXProj && !AF && xproj_decode_skinny(M, N)) || (!AF && !CF && decode_tiles(M, N, K))) {
        SkinnyArgs p{};
        p.A = A; p.lda = lda; p.a_f32 = AF; p.B = (const bf16*)B; p.ldb = ldb; p.C = C; p.ldc = ldc;
        p.M = (int)M; p.N = (int)N; p.K = (int)K;
        return launch_gemm_skinny(p, CF ? kSkinnyStoreF32 : kSkinnyStoreBf16, s);
    }
    if constexpr (ROLE == kGemmXProj && !AF) {
        // x_proj: few output columns (R + 2N), long K; one 64-row tile spans all of N so
        // that every activation row is read once, with a 3-deep ring to cover the latency
        // that four waves per CU leave exposed
        if (K % 64 == 0 && N <= 256) {
            const int sp = fit_slices(splitk_slices((M + 63) / 64, K), M, N, scratch_bytes);
            if (N <= 192) return run_dma<ROLE, 64, 192, 64, 3, 2, 2, CF>(M, N, K, A, lda, B, ldb, C, ldc, s, sp, scratch);
            return run_dma<ROLE, 64, 256, 64, 3, 2, 2, CF>(M, N, K, A, lda, B, ldb, C, ldc, s, sp, scratch);
        }
    }
    if constexpr (!AF) {
        if (K % 32 == 0) return dispatch_dma<ROLE, CF>(M, N, K, A, lda, B, ldb, C, ldc, s, scratch, scratch_bytes);
    }
    // staged path: fp32 A (rounded while staging) or a K tail; short K favours more tiles
    const int64_t big_tiles = ((M + 255) / 256) * ((N + 255) / 256);
    if (big_tiles >= 512 && K > 256) return run_bf16<ROLE, 256, 256, 2, 2, AF, CF>(M, N, K, A, lda, B, ldb, C, ldc, s);
    return run_bf16<ROLE, 128, 128, 2, 2, AF, CF>(M, N, K, A, lda, B, ldb, C, ldc, s);
}

}  // namespace

hipError_t launch_round_bf16_rows(const float* a, int64_t lda, void* o, int64_t M, int K, hipStream_t s) {
    const int64_t n8 = M * (K / 8);
    if (n8 <= 0) return hipSuccess;
    SSM_LAUNCH(round_bf16_rows_kernel, dim3((unsigned)((n8 + 255) / 256)), dim3(256), 0, s, a, lda, (bf16*)o, M, K);
    return hipGetLastError();
}

size_t gemm_splitk_bytes(int64_t M, int64_t N, int64_t K, int a_dt, int b_dt, GemmRole role) {
    // float32 operands on 128x128 tiles (more than the 64 rows of the streamed kernel)
    if (a_dt == SSM_F32 && b_dt == SSM_F32) {
        if (M <= 64 || N == 0 || f32_slices(((M + 127) / 128) * ((N + 127) / 128), K) <= 1) return 0;
        const int sp = f32_slices(((M + 63) / 64) * ((N + 63) / 64), K);
        return sp > 1 ? (size_t)sp * M * N * 4 : 0;
    }
    // mirrors the dispatch below: the DMA paths with bf16 operands and K % 64 == 0
    if (M <= 64 || N == 0 || b_dt != SSM_BF16 || a_dt != SSM_BF16 || K % 64 != 0) return 0;
    int64_t tiles;
    if (role == kGemmXProj && xproj_decode_skinny(M, N)) return 0;
    if (decode_tiles(M, N, K) && role != kGemmXProj) return 0;
    if (role == kGemmXProj && N <= 256) tiles = (M + 63) / 64;
    else if (dma_big_tiles(M, N)) return 0;
    else tiles = ((M + 127) / 128) * ((N + 127) / 128);
    const int sp = splitk_slices(tiles, K);
    return sp > 1 ? (size_t)sp * M * N * 4 : 0;
}

hipError_t launch_gemm_nt(int64_t M, int64_t N, int64_t K, const void* A, int64_t lda, int a_dt, const void* B,
                          int64_t ldb, int b_dt, void* C, int64_t ldc, int c_dt, hipStream_t s, GemmRole role,
                          float* scratch, size_t scratch_bytes) {
    if (M == 0 || N == 0) return hipSuccess;
    if (b_dt == SSM_F32) {
        // up to 64 rows (a decode step): the weight stream in whole lines
        if (M <= 64) {
            const hipError_t e = launch_gemv_f32_stream(role, M, N, K, (const float*)A, lda, (const float*)B, ldb,
                                                        (float*)C, ldc, s);
            if (e != hipErrorNotSupported) return e;
        }
        auto al16 = [](const void* q) { return ((uintptr_t)q & 15) == 0; };
        if (M <= 8 && K % 4 == 0 && lda % 4 == 0 && ldb % 4 == 0 && al16(A) && al16(B)) {
            const dim3 grid((unsigned)((N + 3) / 4));
#define SSM_F32_GEMV(R)                                                                                              \
    case R:                                                                                                          \
        SSM_LAUNCH(gemv_f32_kernel<R>, grid, dim3(256), 0, s, (int)M, (int)N, (int)K, (const float*)A, lda,         \
                   (const float*)B, ldb, (float*)C, ldc);                                                            \
        break;
            switch (role) {
                SSM_F32_GEMV(kGemmInProj)
                SSM_F32_GEMV(kGemmXProj)
                SSM_F32_GEMV(kGemmDtProj)
                SSM_F32_GEMV(kGemmOutProj)
                default: SSM_F32_GEMV(kGemmGeneric)
            }
#undef SSM_F32_GEMV
            return hipGetLastError();
        }
        // prefill sizes on the DMA tiles (float32 rows moved as bytes, run_dma_f32): when the
        // output has few 128x128 tiles (x_proj: 32), K-slices of 64x64 tiles (4 waves of 32x32,
        // a 4-deep ring of 16 KB stages, two workgroups per CU), whose partials are a quarter of
        // those of 128x128 slices for as many workgroups; else the tile shape of least modelled
        // time (f32_tiles)
        {
            const int64_t tm2 = (M + 127) / 128, tn2 = (N + 127) / 128;
            const bool few = f32_slices(tm2 * tn2, K) > 1;
            const int sp = few ? fit_slices(f32_slices(((M + 63) / 64) * ((N + 63) / 64), K), M, N, scratch_bytes) : 1;
            if (K % kF32BK == 0 && (tm2 * tn2 >= 256 || few) && lda % 4 == 0 && ldb % 4 == 0 && al16(A) &&
                al16(B) && al16(C) && 256 * lda * 4 < ((int64_t)1 << 31) && 256 * ldb * 4 < ((int64_t)1 << 31)) {
                const F32Tiles t = few ? kF32Tiles64 : f32_tiles(M, N);
                float* part = sp > 1 ? scratch : nullptr;
                const float* fA = (const float*)A;
                const float* fB = (const float*)B;
                float* fC = (float*)C;
#define SSM_F32_DMA(R)                                                                                         \
    case R:                                                                                                    \
        switch (t) {                                                                                           \
            case kF32Tiles256: return run_dma_f32<R, 256, 256, 2, 2, 4>(M, N, K, fA, lda, fB, ldb, fC, ldc, s); \
            case kF32Tiles256x224: return run_dma_f32<R, 256, 224, 2, 8, 1>(M, N, K, fA, lda, fB, ldb, fC, ldc, s); \
            case kF32Tiles128x224: return run_dma_f32<R, 128, 224, 2, 4, 2, true>(M, N, K, fA, lda, fB, ldb, fC, ldc, s); \
            case kF32Tiles64: return run_dma_f32<R, 64, 64, 4, 2, 2>(M, N, K, fA, lda, fB, ldb, fC, ldc, s, sp, part); \
            default: return run_dma_f32<R, 128, 128, 2, 2, 4>(M, N, K, fA, lda, fB, ldb, fC, ldc, s); \
        }
                switch (role) {
                    SSM_F32_DMA(kGemmInProj)
                    SSM_F32_DMA(kGemmXProj)
                    SSM_F32_DMA(kGemmDtProj)
                    SSM_F32_DMA(kGemmOutProj)
                    default: SSM_F32_DMA(kGemmGeneric)
                }
#undef SSM_F32_DMA
            }
        }
        const int tm = (int)((M + 63) / 64), tn = (int)((N + 63) / 64);
#define SSM_F32_CASE(R)                                                                                             \
    case R:                                                                                                         \
        SSM_LAUNCH(gemm_f32_nt<R>, dim3(tm * tn), dim3(256), 0, s, (int)M, (int)N, (int)K, (const float*)A, \
                           lda, (const float*)B, ldb, (float*)C, ldc, tm, tn);                                      \
        break;
        switch (role) {
            SSM_F32_CASE(kGemmInProj)
            SSM_F32_CASE(kGemmXProj)
            SSM_F32_CASE(kGemmDtProj)
            SSM_F32_CASE(kGemmOutProj)
            default: SSM_F32_CASE(kGemmGeneric)
        }
#undef SSM_F32_CASE
        return hipGetLastError();
    }
    const bool af = a_dt == SSM_F32, cf = c_dt == SSM_F32;
    // the mixer's projections use one operand combination each
    switch (role) {
        case kGemmInProj:
            if (!af && !cf) return dispatch_bf16<kGemmInProj, false, false>(M, N, K, A, lda, B, ldb, C, ldc, s, scratch, scratch_bytes);
            break;
        case kGemmXProj:
            if (!af && cf) return dispatch_bf16<kGemmXProj, false, true>(M, N, K, A, lda, B, ldb, C, ldc, s, scratch, scratch_bytes);
            break;
        case kGemmDtProj:
            if (af && !cf) return dispatch_bf16<kGemmDtProj, true, false>(M, N, K, A, lda, B, ldb, C, ldc, s, scratch, scratch_bytes);
            if (!af && !cf) return dispatch_bf16<kGemmDtProj, false, false>(M, N, K, A, lda, B, ldb, C, ldc, s, scratch, scratch_bytes);
            break;
        case kGemmOutProj:
            if (!af && !cf) return dispatch_bf16<kGemmOutProj, false, false>(M, N, K, A, lda, B, ldb, C, ldc, s, scratch, scratch_bytes);
            break;
        default:
            break;
    }
    if (af && cf) return dispatch_bf16<kGemmGeneric, true, true>(M, N, K, A, lda, B, ldb, C, ldc, s, scratch, scratch_bytes);
    if (af) return dispatch_bf16<kGemmGeneric, true, false>(M, N, K, A, lda, B, ldb, C, ldc, s, scratch, scratch_bytes);
    if (cf) return dispatch_bf16<kGemmGeneric, false, true>(M, N, K, A, lda, B, ldb, C, ldc, s, scratch, scratch_bytes);
    return dispatch_bf16<kGemmGeneric, false, false>(M, N, K, A, lda, B, ldb, C, ldc, s, scratch, scratch_bytes);
}

}  // namespace ssm
