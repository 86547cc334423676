/*
 * ssm_shard.h - C ABI of the selective-SSM (Mamba-1) mixer on one tensor-parallel
 * channel shard, for AMD Instinct MI355X (gfx950).
 *
 * Source: "Scaling State-Space Models on Multiple GPUs with Tensor Parallelism".
 *   - Section II-B / Fig. 1: the mixer's op order (in_proj, split into SSM and gate
 *     paths, short channel-separable convolution, projection to packed Delta/B/C,
 *     discretisation with per-channel A, state update with D skip, gate, out_proj).
 *   - Section IV-A: the SSM cache = final recurrent state + last K-1 convolution
 *     inputs per sequence, sharded by channel, written by prefill and read and
 *     advanced by decode without rescanning the prompt.
 *   - Section IV-B: channel-wise splitting; each rank owns a contiguous channel range;
 *     exactly two reductions per block: after x_proj and at the residual boundary.
 *   - Section IV-C: the packed [delta | B | C] parameters are unpacked by column
 *     range; Delta is sharded with channels, B and C are complete on every rank after
 *     the first reduction, A and D are per channel and local.
 *
 * Conventions (all entry points):
 *   - Every tensor argument is DEVICE memory owned by the caller, row-major with the
 *     last dimension contiguous, 16-byte aligned. The library never allocates; the
 *     caller provides a workspace of at least the size the *_workspace_bytes query
 *     returns. Inputs are never modified; cache pools are updated in place.
 *   - "act" tensors hold the activation dtype of the descriptor (SSM_BF16 or SSM_F32).
 *   - Calls are asynchronous on the given HIP stream (0 = the null stream).
 *   - Return value: SSM_OK (0) or a negative SSM_E_* code. All argument checks happen
 *     on the host before anything is enqueued; a failed check enqueues nothing.
 *     ssm_last_error() gives a message for the calling thread's last failure.
 *   - Per-sequence metadata (cu_seqlens, cache_slot, has_initial_state) is DEVICE
 *     int32 memory so that calls can be enqueued without host round trips. Kernels
 *     never index out of range with it: an out-of-range slot or a non-monotone
 *     cu_seqlens entry makes the affected work a no-op and sets a bit in the
 *     workspace status word (SSM_STATUS_*), read with ssm_shard_take_status().
 *     ssm_shard_check_meta_host() validates host copies completely (including
 *     duplicate slots, which the kernels cannot detect; duplicates in one call race).
 *   - Cache layout: conv_pool [num_slots][E][K-1] act dtype, oldest input first (empty,
 *     and the pointer may be null, when K = 1); ssm_pool [num_slots][E][N] float32.
 *     Slots not named in a call stay bit-identical.
 */
#ifndef SSM_SHARD_H
#define SSM_SHARD_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SSM_SHARD_ABI_VERSION 1

/* Return codes. */
#define SSM_OK 0
#define SSM_E_INVAL (-1)     /* bad descriptor, shape, dtype or null pointer      */
#define SSM_E_ALIGN (-2)     /* pointer or leading dimension not aligned          */
#define SSM_E_WORKSPACE (-3) /* workspace smaller than the size query returned    */
#define SSM_E_SLOT (-4)      /* cache slot out of range or duplicated (host check)*/
#define SSM_E_SEQLENS (-5)   /* cu_seqlens not 0 = c0 <= c1 <= ... = T (host check)*/
#define SSM_E_HIP (-6)       /* a HIP runtime call failed                          */

/* Bits of the workspace status word, set by kernels that met bad device metadata. */
#define SSM_STATUS_BAD_SLOT 1
#define SSM_STATUS_BAD_SEQLENS 2

/* Storage dtype of activations and act-typed weights. */
typedef enum ssm_dtype { SSM_F32 = 0, SSM_BF16 = 1 } ssm_dtype_t;

/* Shape of one layer and of the shard this rank owns (Section IV-B). The shard owns
 * channels [shard_index * d_inner_shard, (shard_index + 1) * d_inner_shard).
 * Requirements: d_inner_shard * shard_count == d_inner_total; d_state == 16;
 * d_conv in [1, 4]; d_model and dt_rank multiples of 16; d_inner_shard a multiple
 * of 64 (the scan and decode kernels give each 64-lane wave 64 whole channels). */
typedef struct ssm_shard_desc {
    int32_t d_model;        /* residual width                                   */
    int32_t d_inner_total;  /* E_tot, intermediate channels of the whole layer  */
    int32_t d_inner_shard;  /* E, channels of this shard                        */
    int32_t d_state;        /* N, states per channel                            */
    int32_t dt_rank;        /* R, width of the low-rank step-size input         */
    int32_t d_conv;         /* K, convolution taps                              */
    int32_t shard_index;    /* this rank                                        */
    int32_t shard_count;    /* P, channel-split degree                          */
    int32_t act_dtype;      /* ssm_dtype_t                                      */
} ssm_shard_desc_t;

/* One shard's weights (device pointers), already sliced to the shard's channels.
 *   in_proj_w  [2E][d_model] act: rows 0..E-1 feed the SSM path, rows E..2E-1 the gate
 *   conv_w     [E][K] act, conv_b [E] act (tap K-1 multiplies the current token)
 *   x_proj_w   [R+2N][E] act: output columns are [delta | B | C]
 *   dt_proj_w  [E][R] act, dt_proj_b [E] float32
 *   A_log      [E][N] float32 (A = -exp(A_log)), D [E] float32
 *   out_proj_w [d_model][E] act */
typedef struct ssm_shard_weights {
    const void* in_proj_w;
    const void* conv_w;
    const void* conv_b;
    const void* x_proj_w;
    const void* dt_proj_w;
    const void* out_proj_w;
    const float* dt_proj_b;
    const float* A_log;
    const float* D;
} ssm_shard_weights_t;

/* Packed variable-length batch (device int32 arrays).
 *   cu_seqlens [nseq+1]: sequence i occupies packed tokens [cu_seqlens[i], cu_seqlens[i+1])
 *   cache_slot [nseq]: pool slot of sequence i
 *   has_initial_state [nseq]: 1 = continue from the slot's cached conv history and
 *     state (a chunk of a longer prompt), 0 = start from zeros. */
typedef struct ssm_seq_meta {
    const int32_t* cu_seqlens;
    const int32_t* cache_slot;
    const int32_t* has_initial_state;
    int32_t nseq;
} ssm_seq_meta_t;

/* ---------------------------------------------------------------- housekeeping */
int ssm_shard_abi_version(void);
/* Message for the calling thread's most recent failure ("" if none). */
const char* ssm_last_error(void);
/* Checks a descriptor; SSM_OK or SSM_E_INVAL. */
int ssm_shard_check_desc(const ssm_shard_desc_t* desc);
/* Host-side check of HOST copies of the metadata: cu_seqlens[0] == 0, non-decreasing,
 * cu_seqlens[nseq] == T; every slot in [0, num_slots) and no slot repeated;
 * has_initial_state entries 0 or 1. Returns SSM_OK, SSM_E_SEQLENS, SSM_E_SLOT or SSM_E_INVAL. */
int ssm_shard_check_meta_host(const int32_t* cu_seqlens, const int32_t* cache_slot,
                              const int32_t* has_initial_state, int32_t nseq, int64_t T,
                              int32_t num_slots);

/* Workspace sizes. A prefill workspace serves every call with T <= max_tokens and
 * nseq <= max_seqs; a decode workspace serves batches up to max_batch. */
int ssm_shard_prefill_workspace_bytes(const ssm_shard_desc_t* desc, int64_t max_tokens,
                                      int32_t max_seqs, size_t* bytes);
int ssm_shard_decode_workspace_bytes(const ssm_shard_desc_t* desc, int32_t max_batch, size_t* bytes);
/* Zero the workspace status word (call once after allocating a workspace). Calls that
 * share a workspace must not overlap in time. */
int ssm_shard_workspace_init(void* ws, size_t ws_bytes, hipStream_t stream);
/* Synchronise the stream, read the status word into *status and clear it. */
int ssm_shard_take_status(void* ws, size_t ws_bytes, int32_t* status, hipStream_t stream);

/* ------------------------------------------------------------------ prefill
 * ssm_shard_prefill: the whole shard over a packed batch of T tokens.
 *   x [T][d_model] act -> y_partial [T][d_model] act, this shard's out_proj partial sum
 *   (the second reduction, at the residual boundary, is the caller's).
 * Writes conv_pool[slot] and ssm_pool[slot] of every sequence in meta.
 * The first reduction (x_proj sum over ranks) is taken as the identity: exact when
 * shard_count == 1; with several shards use the two stages below. */
int ssm_shard_prefill(const ssm_shard_desc_t* desc, const ssm_shard_weights_t* w,
                      const void* x, int64_t T, const ssm_seq_meta_t* meta,
                      void* conv_pool, float* ssm_pool, int32_t num_slots,
                      void* y_partial, void* ws, size_t ws_bytes, hipStream_t stream);

/* Stage 1: in_proj, causal conv1d + SiLU (writes conv_pool), x_proj.
 *   x_dbl_partial [T][R+2N] float32 out: this shard's partial x_proj output.
 * Keeps xz and u in ws for stage 2 (pass the same ws, T and meta to stage 2). */
int ssm_shard_prefill_stage1(const ssm_shard_desc_t* desc, const ssm_shard_weights_t* w,
                             const void* x, int64_t T, const ssm_seq_meta_t* meta,
                             void* conv_pool, int32_t num_slots, float* x_dbl_partial,
                             void* ws, size_t ws_bytes, hipStream_t stream);
/* Stage 2: from the x_proj output summed over all shards (x_dbl [T][R+2N] float32):
 * dt_proj, selective scan with D skip and gate (writes ssm_pool), out_proj. */
int ssm_shard_prefill_stage2(const ssm_shard_desc_t* desc, const ssm_shard_weights_t* w,
                             const float* x_dbl, int64_t T, const ssm_seq_meta_t* meta,
                             float* ssm_pool, int32_t num_slots, void* y_partial,
                             void* ws, size_t ws_bytes, hipStream_t stream);

/* ------------------------------------------------------------------- decode
 * One token for each of `batch` sequences, advancing their cached history and state
 * in place (Section IV-A). cache_slot [batch] device int32, distinct.
 *   x_t [batch][d_model] act -> y_partial [batch][d_model] act. */
int ssm_shard_decode_step(const ssm_shard_desc_t* desc, const ssm_shard_weights_t* w,
                          const void* x_t, int32_t batch, const int32_t* cache_slot,
                          void* conv_pool, float* ssm_pool, int32_t num_slots,
                          void* y_partial, void* ws, size_t ws_bytes, hipStream_t stream);
int ssm_shard_decode_stage1(const ssm_shard_desc_t* desc, const ssm_shard_weights_t* w,
                            const void* x_t, int32_t batch, const int32_t* cache_slot,
                            void* conv_pool, int32_t num_slots, float* x_dbl_partial,
                            void* ws, size_t ws_bytes, hipStream_t stream);
int ssm_shard_decode_stage2(const ssm_shard_desc_t* desc, const ssm_shard_weights_t* w,
                            const float* x_dbl, int32_t batch, const int32_t* cache_slot,
                            float* ssm_pool, int32_t num_slots, void* y_partial,
                            void* ws, size_t ws_bytes, hipStream_t stream);

/* Decode step for callers that cannot allocate (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc): the same computation and kernels as
 * ssm_shard_decode_step, with its workspace taken from a static device array of
 * SSM_NOALLOC_SCRATCH_BYTES that the library holds on each GPU it runs on until the
 * process ends. The call allocates nothing (leave ssm_timing_enable off: timed launches
 * may create events). A batch whose workspace would exceed the array (the size
 * ssm_shard_decode_workspace_bytes reports) returns SSM_E_WORKSPACE and enqueues nothing.
 * The array is shared by every call on one GPU, and calls that overlap in time on one
 * GPU race; run them on one stream or otherwise in order. Bad device slots still never
 * cause an out-of-range access, but their status bits are not reported here (validate
 * slots with ssm_shard_check_meta_host, or use ssm_shard_decode_step to read them).
 * The stream must belong to the current device. */
#define SSM_NOALLOC_SCRATCH_BYTES (32u << 20)
int ssm_shard_decode_step_noalloc(const ssm_shard_desc_t* desc, const ssm_shard_weights_t* w,
                                  const void* x_t, int32_t batch, const int32_t* cache_slot,
                                  void* conv_pool, float* ssm_pool, int32_t num_slots,
                                  void* y_partial, hipStream_t stream);

/* ------------------------------------------------------------------ utilities
 * Channel splitter (Section IV-B): copy this shard's slices of full-width weights
 * (full: same fields at full width, E_tot channels) into caller-allocated shard
 * buffers (out: fields point to writable device memory of the shard shapes).
 * in_proj's x rows and z rows are sliced separately; x_proj and out_proj by column. */
int ssm_shard_slice_weights(const ssm_shard_desc_t* desc, const ssm_shard_weights_t* full,
                            const ssm_shard_weights_t* out, hipStream_t stream);
/* dst[i] += src[i] for i < n (float32): the x_proj exchange when all shards run on one GPU. */
int ssm_reduce_add_f32(float* dst, const float* src, int64_t n, hipStream_t stream);

/* --------------------------------------------------- quantized exchange
 * Section IV-D: the two remaining AllReduces (the x_proj output, fp32, and the out_proj
 * partial, act dtype) may carry a lower precision than the computation -- FP16 in the
 * paper -- and are converted back for what follows. One exchange of P partials is an
 * encode on every rank and, on the receiver, a decode of each payload added into an
 * fp32 sum in rank order (an all-gather of payloads followed by a local reduction).
 *   SSM_CODEC_F16, SSM_CODEC_BF16: element-wise rounding (ties to even), 2 bytes/value;
 *     values beyond the half range become infinities, as IEEE conversion does.
 *   SSM_CODEC_FP8_E4M3: OCP FP8 E4M3 of x * (448 / max|row|), 1 byte/value, one fp32
 *     scale per row (amax / 448); SSM_CODEC_INT8: round-half-even of x * (127 / max|row|)
 *     clamped to [-127, 127], one fp32 scale per row (amax / 127). A zero row has scale 0.
 * Payload layout (device memory, caller-owned): scaled codecs first hold the [rows] fp32
 * scales, padded to a multiple of 256 bytes, then the [rows][cols] codes, dense; the
 * 2-byte codecs hold only the codes. Inputs must be finite. cols, ld_src and ld_acc are
 * multiples of 8 and the pointers 16-byte aligned (else SSM_E_ALIGN); a payload smaller
 * than the size query returns SSM_E_WORKSPACE. Stream-ordered, no allocation. */
typedef enum ssm_codec { SSM_CODEC_F16 = 0, SSM_CODEC_BF16 = 1, SSM_CODEC_FP8_E4M3 = 2, SSM_CODEC_INT8 = 3 } ssm_codec_t;
int ssm_exchange_payload_bytes(int32_t codec, int64_t rows, int64_t cols, size_t* bytes);
/* payload <- encode(src), src [rows][cols] of src_dtype (ssm_dtype_t) with row stride ld_src */
int ssm_exchange_encode(int32_t codec, const void* src, int32_t src_dtype, int64_t rows, int64_t cols,
                        int64_t ld_src, void* payload, size_t payload_bytes, hipStream_t stream);
/* acc [rows][cols] fp32 (row stride ld_acc) = decode(payload) (+ acc when accumulate != 0) */
int ssm_exchange_decode_accumulate(int32_t codec, const void* payload, size_t payload_bytes, int64_t rows,
                                   int64_t cols, float* acc, int64_t ld_acc, int32_t accumulate,
                                   hipStream_t stream);

/* ------------------------------------------------------- stage operators
 * The kernels the entry points above are built from, exposed for kernel-level checks.
 *
 * C[M][N] = A[M][K] * B[N][K]^T, float32 accumulation. a_dtype, b_dtype, c_dtype are
 * ssm_dtype_t. With b_dtype == SSM_BF16 the product runs on bf16 matrix cores and a
 * float32 A is rounded to bf16 (ties to even) as it is loaded; with b_dtype == SSM_F32
 * both operands must be float32. K, lda, ldb multiples of 8; ldc a multiple of 4. */
int ssm_gemm_nt(int64_t M, int64_t N, int64_t K, const void* A, int64_t lda, int32_t a_dtype,
                const void* B, int64_t ldb, int32_t b_dtype, void* C, int64_t ldc, int32_t c_dtype,
                hipStream_t stream);
/* The same product on the kernel instance and tile policy of one projection (role: 0
 * generic, 1 in_proj, 2 x_proj, 3 dt_proj, 4 out_proj), as the prefill runs it. Outputs
 * with fewer tiles than the GPU has compute units and a long K are computed split-K: the
 * K-slices' float32 partials go to scratch (device, the caller's; ssm_gemm_splitk_bytes
 * gives its size, 0 when the shape is not split) and a second kernel adds them in slice
 * order. With less scratch than that (or none) the product runs unsplit. */
int ssm_gemm_splitk_bytes(int64_t M, int64_t N, int64_t K, int32_t a_dtype, int32_t b_dtype, int32_t role,
                          size_t* bytes);
int ssm_gemm_nt_role(int64_t M, int64_t N, int64_t K, const void* A, int64_t lda, int32_t a_dtype, const void* B,
                     int64_t ldb, int32_t b_dtype, void* C, int64_t ldc, int32_t c_dtype, int32_t role,
                     float* scratch, size_t scratch_bytes, hipStream_t stream);
/* Causal depthwise conv1d + SiLU over a packed batch: reads the SSM half of
 * xz [T][2E] (columns 0..E-1), writes u [T][E] act and the new conv history. */
int ssm_conv1d_silu(const ssm_shard_desc_t* desc, const ssm_shard_weights_t* w, const void* xz,
                    int64_t T, const ssm_seq_meta_t* meta, void* conv_pool, int32_t num_slots,
                    void* u, void* ws, size_t ws_bytes, hipStream_t stream);
/* Selective scan: Delta = softplus(dt + dt_proj_b), h <- exp(Delta*A) h + Delta*B*u,
 * y = C.h + D*u, g = y * SiLU(z). u, dt [T][E] act; z = columns E..2E-1 of xz [T][2E];
 * B, C = columns R..R+N-1 and R+N..R+2N-1 of x_dbl [T][R+2N] float32.
 * Writes g [T][E] act and ssm_pool[slot] of every sequence. */
int ssm_selective_scan(const ssm_shard_desc_t* desc, const ssm_shard_weights_t* w,
                       const void* u, const void* dt, const void* xz, const float* x_dbl,
                       int64_t T, const ssm_seq_meta_t* meta, float* ssm_pool, int32_t num_slots,
                       void* g, void* ws, size_t ws_bytes, hipStream_t stream);
/* Decode: shift each sequence's cached window by the new token (column c of xz) and
 * convolve: u [batch][E]; conv_pool updated in place. */
int ssm_decode_conv(const ssm_shard_desc_t* desc, const ssm_shard_weights_t* w, const void* xz,
                    int32_t batch, const int32_t* cache_slot, void* conv_pool, int32_t num_slots,
                    void* u, void* ws, size_t ws_bytes, hipStream_t stream);
/* Decode: one recurrence step per sequence on ssm_pool[slot] in place, with D skip and
 * gate; same operand layout as ssm_selective_scan with T = batch. */
int ssm_decode_ssm(const ssm_shard_desc_t* desc, const ssm_shard_weights_t* w, const void* u,
                   const void* dt, const void* xz, const float* x_dbl, int32_t batch,
                   const int32_t* cache_slot, float* ssm_pool, int32_t num_slots, void* g,
                   void* ws, size_t ws_bytes, hipStream_t stream);

/* ------------------------------------------------------- Mamba-2 (SSD) shard
 * Section II-A and Section IV-E: Mamba-2 keeps the mixer pipeline (projection,
 * convolution, state update, gating, output projection) with a multi-head state whose
 * update maps onto matrix products; the split is by heads and reuses the same cache and
 * exchange principles. Per head h (scalar decay, headdim P, N states per row):
 *   Delta_t = softplus(dt_t + dt_bias_h);  S_t = exp(-exp(A_log_h) Delta_t) S_{t-1} + Delta_t x_t B_t^T
 *   y_t = S_t C_t + D_h x_t;  g_t = y_t * SiLU(z_t);  g_norm = g / sqrt(mean_group(g^2) + 1e-5) * norm_w
 * with B_t, C_t of the head's group, and y_partial = out_proj(g_norm).
 * Shard: H = nheads_total / shard_count heads, E = H * headdim channels; B/C groups are
 * split (Gs = ngroups_total / shard_count) when ngroups_total is a multiple of
 * shard_count, else every shard holds all of them (Gs = ngroups_total). The gated
 * norm's group is d_inner / ngroups_total channels: stage 1 ends with each shard's
 * partial sum of g^2 per token and norm group [T][ngroups_total] (float32); the caller
 * sums these over shards (the exchange; identity for one shard) and stage 2 normalises
 * and projects, reading the g that stage 1 left in the same workspace.
 * Requirements: headdim == 64, d_state == 128, act_dtype SSM_BF16, nheads_total a
 * multiple of shard_count and of ngroups_total, H a multiple of 8, d_model a multiple
 * of 16, 2 <= d_conv <= 4. Caches: conv [S][E + 2 Gs N][d_conv - 1] act (oldest first,
 * channels x | B | C), state [S][H][64][128] float32. */
typedef struct ssm2_shard_desc {
    int32_t d_model, nheads_total, headdim, d_state, ngroups_total, d_conv;
    int32_t shard_index, shard_count;
    int32_t act_dtype;
} ssm2_shard_desc_t;
/* Shard weights (device, caller-owned). in_proj rows in order z (E), x (E), B (Gs*N),
 * C (Gs*N), dt (H); conv channels x (E), B (Gs*N), C (Gs*N). A full-width layer uses the
 * same struct with the full sizes (shard_count 1) and is the input of the splitter. */
typedef struct ssm2_shard_weights {
    const void* in_proj_w;   /* [2E + 2 Gs N + H][d_model] act */
    const void* conv_w;      /* [E + 2 Gs N][d_conv] act */
    const void* conv_b;      /* [E + 2 Gs N] act */
    const void* out_proj_w;  /* [d_model][E] act */
    const float* dt_bias;    /* [H] */
    const float* A_log;      /* [H] */
    const float* D;          /* [H] */
    const float* norm_w;     /* [E] */
} ssm2_shard_weights_t;
int ssm2_shard_check_desc(const ssm2_shard_desc_t* desc);
int ssm2_shard_prefill_workspace_bytes(const ssm2_shard_desc_t* desc, int64_t max_tokens, int32_t max_seqs,
                                       size_t* bytes);
int ssm2_shard_decode_workspace_bytes(const ssm2_shard_desc_t* desc, int32_t max_batch, size_t* bytes);
/* Copy this shard's slices out of full-width weights (the layout above with shard_count 1). */
int ssm2_shard_slice_weights(const ssm2_shard_desc_t* desc, const ssm2_shard_weights_t* full,
                             const ssm2_shard_weights_t* out, hipStream_t stream);
/* Packed prefill, x [T][d_model] act; metadata as for ssm_shard_prefill. */
int ssm2_shard_prefill_stage1(const ssm2_shard_desc_t* desc, const ssm2_shard_weights_t* w, const void* x,
                              int64_t T, const ssm_seq_meta_t* meta, void* conv_pool, float* ssm_pool,
                              int32_t num_slots, float* sumsq_partial, void* ws, size_t ws_bytes,
                              hipStream_t stream);
int ssm2_shard_prefill_stage2(const ssm2_shard_desc_t* desc, const ssm2_shard_weights_t* w, const float* sumsq,
                              int64_t T, void* y_partial, void* ws, size_t ws_bytes, hipStream_t stream);
/* One token per sequence, x_t [batch][d_model]; cache_slot [batch] device int32. */
int ssm2_shard_decode_stage1(const ssm2_shard_desc_t* desc, const ssm2_shard_weights_t* w, const void* x_t,
                             int32_t batch, const int32_t* cache_slot, void* conv_pool, float* ssm_pool,
                             int32_t num_slots, float* sumsq_partial, void* ws, size_t ws_bytes,
                             hipStream_t stream);
int ssm2_shard_decode_stage2(const ssm2_shard_desc_t* desc, const ssm2_shard_weights_t* w, const float* sumsq,
                             int32_t batch, void* y_partial, void* ws, size_t ws_bytes, hipStream_t stream);

/* ------------------------------------------------------------ the layer around the mixer
 * Section II-B: after out_proj the block returns to the residual stream by adding the
 * mixer's output to the incoming hidden states. Under tensor parallelism that output is
 * the sum over ranks of the out_proj partials (Section IV-B's second reduction), so the
 * add follows that exchange. In front of every mixer the residual is RMS-normalised with
 * a per-channel weight (pre-norm), and a final RMSNorm follows the last layer. The
 * residual stream is float32. */

/* residual = base + (parts[0] + ... + parts[n_parts-1]), the parts summed in float32 in
 * that order; normed = residual / sqrt(mean over the row of residual^2 + eps) * norm_w.
 *   base      [T][d] of base_dtype (SSM_F32 or SSM_BF16); may equal residual (in place)
 *   parts     host array of n_parts (0..8) device pointers, each [T][d] of parts_dtype
 *             (the ranks' out_proj partials, or one already reduced sum)
 *   residual  [T][d] float32, written;  norm_w [d] float32;  normed [T][d] of normed_dtype
 * Rows are contiguous. d must be a multiple of 8 and at most 8192. Device memory is the
 * caller's; nothing else is modified. SSM_E_INVAL for bad sizes, dtypes, null pointers or
 * a base that partially overlaps residual; SSM_E_ALIGN for pointers not 16-byte aligned. */
int ssm_residual_rmsnorm(const void* base, int32_t base_dtype, const void* const* parts, int32_t n_parts,
                         int32_t parts_dtype, float* residual, const float* norm_w, float eps, void* normed,
                         int32_t normed_dtype, int64_t T, int32_t d, hipStream_t stream);

/* Falcon-Mamba (Section IV-E names it as using the same selective SSM mixer; its model
 * normalises the token-dependent fields): on the reduced x_proj output x_dbl [T][ld]
 * float32, in place, the column ranges [0,R) (delta), [R,R+N) (B) and [R+N,R+2N) (C) are
 * each divided by sqrt(mean of their squares + eps); no weight. It runs after the first
 * exchange and before stage 2 (prefill or decode). SSM_E_INVAL for ld < R + 2N or eps <= 0. */
int ssm_bcdt_rmsnorm(float* x_dbl, int64_t T, int32_t R, int32_t N, int64_t ld, float eps, hipStream_t stream);

/* A stack of n_layers mixer layers at full width on one GPU (layer.shard_count == 1: both
 * exchanges are identities; a split stack is composed from the per-layer calls and the
 * caller's exchanges). With r_0 = x:
 *   h = RMSNorm_l(r_l) (act dtype);  [stage 1;  Falcon-Mamba norms if bcdt_eps > 0;  stage 2]
 *   r_{l+1} = r_l + y_l;  out = RMSNorm_final(r_L) (act dtype).
 * layers, norm_w, conv_pools and ssm_pools are host arrays of n_layers entries holding
 * device pointers (norm weights [d_model] float32; pools as for the one-layer calls, one
 * pair per layer, all with num_slots slots); meta, cache slots and errors as for
 * ssm_shard_prefill / ssm_shard_decode_step. x, x_t and out are [rows][d_model] act.
 * The workspace queries give the size for up to max_tokens / max_batch rows. */
typedef struct ssm_stack_desc {
    ssm_shard_desc_t layer;   /* every layer's mixer; shard_count 1 */
    int32_t n_layers;
    float norm_eps;           /* RMSNorm eps, > 0 (1e-5 for the Mamba models) */
    float bcdt_eps;           /* > 0: Falcon-Mamba's delta/B/C norms with this eps (1e-6); 0: none */
} ssm_stack_desc_t;
int ssm_stack_prefill_workspace_bytes(const ssm_stack_desc_t* desc, int64_t max_tokens, int32_t max_seqs,
                                      size_t* bytes);
int ssm_stack_decode_workspace_bytes(const ssm_stack_desc_t* desc, int32_t max_batch, size_t* bytes);
int ssm_stack_prefill(const ssm_stack_desc_t* desc, const ssm_shard_weights_t* layers, const float* const* norm_w,
                      const float* final_norm_w, const void* x, int64_t T, const ssm_seq_meta_t* meta,
                      void* const* conv_pools, float* const* ssm_pools, int32_t num_slots, void* out, void* ws,
                      size_t ws_bytes, hipStream_t stream);
int ssm_stack_decode_step(const ssm_stack_desc_t* desc, const ssm_shard_weights_t* layers,
                          const float* const* norm_w, const float* final_norm_w, const void* x_t, int32_t batch,
                          const int32_t* cache_slot, void* const* conv_pools, float* const* ssm_pools,
                          int32_t num_slots, void* out, void* ws, size_t ws_bytes, hipStream_t stream);

/* ------------------------------------------------------------ measurement
 * Per-kernel device time, for benchmarks and profiles only. While enabled, every kernel
 * the library launches from the calling thread is launched with hipExtLaunchKernel and
 * a start/stop event pair bound to that dispatch. A dispatch's reading can include time
 * the GPU spent waiting for the host to submit it (when the queue has drained) or for
 * unfinished work ahead of it, so sample few launches (every k-th) to keep the queue full.
 * Leave timing off in production (each timed launch takes two events). Launches on a
 * stream under graph capture are not timed. */
typedef struct ssm_kernel_time {
    char name[48];       /* kernel role, e.g. "prefill.in_proj", "decode.state_update" */
    int64_t launches;    /* launches recorded since the last collection */
    double total_ms;     /* summed kernel execution time, begin to end of each dispatch */
} ssm_kernel_time_t;
/* on: 0 to stop, 1 to time every launch, k > 1 to time every k-th launch of each kernel
 * name (the first included), which keeps the per-launch event cost, about 5 us on a
 * decode-sized kernel, off all but one launch in k; negative: SSM_E_INVAL. only: NULL to
 * time every kernel, else the one kernel name to time. */
int ssm_timing_enable(int32_t on, const char* only);
/* Waits for the recorded events, sums time per kernel name into out[0 .. *count), at
 * most max entries, and forgets the records. SSM_E_HIP if an event could not be read. */
int ssm_timing_collect(ssm_kernel_time_t* out, int32_t max, int32_t* count);

#ifdef __cplusplus
}
#endif
#endif /* SSM_SHARD_H */
