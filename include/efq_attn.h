/*
 * efq_attn.h -- C ABI of the EFQ-Softmax attention forward for AMD Instinct
 * MI355X (gfx950).
 *
 * The operation is single-head attention O = softmax(Q K^T * scale + M) V,
 * computed tile by tile with the online recurrence of the paper "EFQ-Softmax:
 * Exp-Free Quantization for Softmax" (arXiv 2609.09721), Algorithm 2: the row
 * maximum update, Eq. (rowmax-update); the rescaling factor, Eq. (alpha); the
 * numerator and denominator updates, Eqs. (numerator-basic) and
 * (denominator-basic), both fed by the same block-scaled E2M1 probability
 * operand; and the final division of Sec. III-A.  The probability operand of
 * each 32-key microscaling block comes from Algorithm 1: an exponent-only
 * (E8M0) scale from the block maximum, Eq. (k-rule), and non-negative E2M1
 * codes from the affine rule of Eq. (d8-index) on the residual of Eq. (z-def).
 * V enters the P~V product as MXFP4 (E2M1 codes with one E8M0 scale per 32
 * keys and head-dim column), the low-bit value path of Eq. (numerator-lowbit).
 *
 * Conventions for every entry point
 *  - Tensors are device pointers, contiguous, in BSHD order:
 *      q   [batch][seq_q][heads_q][head_dim]   bf16
 *      k,v [batch][seq_k][heads_kv][head_dim]  bf16
 *      out [batch][seq_q][heads_q][head_dim]   fp32
 *    All device pointers must be 16-byte aligned.  Query head h reads
 *    key/value head h / (heads_q / heads_kv) (grouped-query attention).
 *  - causal != 0 requires seq_q == seq_k; key t is visible to query i iff
 *    t <= i.  Otherwise every key is visible.
 *  - Supported: head_dim 64 or 128, heads_q % heads_kv == 0, any seq >= 1
 *    (ragged tails are masked).  batch * heads_q * ceil(seq_q / 128) must fit
 *    in a 32-bit grid.
 *  - Calls are asynchronous on `stream` (a hipStream_t; NULL = the default
 *    stream) and never synchronise the host (efq_calibrate excepted).  The
 *    caller owns every buffer;
 *    the library keeps no allocation beyond its code objects, except that the
 *    convenience entry points without a workspace argument (and the _ex,
 *    lowbit_ex and calibrate entry points when given no workspace) take one
 *    stream-ordered allocation for their scratch (V~; Q^, K^ and V~; the
 *    calibration buffers) and release it on the same stream.
 *  - Every argument is validated before any HIP call: on error nothing is
 *    enqueued and a negative status is returned.  A failed launch returns
 *    EFQ_EHIP.  efq_strerror() gives a thread-local message for the last
 *    failure of the calling thread.  Calls on different streams may run
 *    concurrently.
 *  - NaN or infinite inputs are not supported: the outputs are then
 *    unspecified, but the call does not fault.
 */
#ifndef EFQ_ATTN_H
#define EFQ_ATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef void *efq_stream_t; /* a hipStream_t */

typedef struct efq_shape {
    int batch, seq_q, seq_k, heads_q, heads_kv, head_dim;
} efq_shape;

/* Affine code parameters (tau, h) of Eq. (d8-index), fixed after the offline
 * calibration of Sec. III-C.  The operating points of Sec. IV-A: */
typedef struct efq_params {
    float tau, h;
} efq_params;
#define EFQ_TAU_MEAN (-3.06f)    /* EFQ-Softmax-Mean (default)  */
#define EFQ_H_MEAN 2.30f
#define EFQ_TAU_MMLU (-2.90f)    /* EFQ-Softmax-MMLU            */
#define EFQ_H_MMLU 2.00f
#define EFQ_TAU_BALANCE (-2.10f) /* EFQ-Softmax-Balance         */
#define EFQ_H_BALANCE 2.70f
/* EFQ-Softmax-LUT (Sec. II-D): tau16 = log(1/24), h16 = 14 / log 24 */
#define EFQ_TAU_LUT (-3.17805383f)
#define EFQ_H_LUT 4.40521173f

/* Probability-stage variants (the "P-gen" policy). */
enum efq_pgen_kind {
    EFQ_PGEN_EFQ = 0,  /* Alg. 1: E8M0 from the block max, affine E2M1 codes   */
    EFQ_PGEN_EXPQ = 1, /* exp-then-quantize baseline, Eq. (post-softmax-path):
                          fp32 exp, then OCP MXFP4 (scale floor(log2 amax)-2,
                          round to nearest even, saturating)                 */
    EFQ_PGEN_LUT = 2,  /* EFQ-Softmax-LUT, Sec. II-D: 16-level index, C16 fold */
    EFQ_PGEN_NOOP = 3, /* timing control only: a constant operand, no P-gen
                          work; its output is meaningless                    */
    EFQ_PGEN_EXPQ6 = 4 /* exp-then-quantize with the "scale6" MXFP4 rule of
                          the comparison rows of Sec. IV: fp32 exp, scale
                          2^ceil(log2(amax / 6)) (amax / scale in (3, 6], so
                          nothing saturates), E2M1 round to nearest even   */
};

enum efq_status {
    EFQ_OK = 0,
    EFQ_EINVAL = -1,       /* bad argument (null pointer, size, alignment)    */
    EFQ_EUNSUPPORTED = -2, /* valid but unsupported (head_dim, causal shape)  */
    EFQ_EWORKSPACE = -3,   /* workspace missing or too small                  */
    EFQ_EHIP = -4          /* HIP runtime error, or no usable gfx950 device    */
};

/* ---------------------------------------------------------------------------
 * V~ workspace: V quantised to MXFP4 along the key axis (the low-bit value
 * operand of Eq. numerator-lowbit; OCP MX rule: E8M0 exponent
 * floor(log2 amax) - 2 per 32 keys and column, E2M1 codes rounded to nearest
 * even with saturation, sign bit = sign of the bf16 input).  Layout, with
 * nb = 2 * ceil(seq_k / 64) key blocks (blocks past seq_k hold zeros):
 *   codes  [batch][heads_kv][nb][head_dim][16 bytes]  32 keys per 16 bytes
 *   scales [batch][heads_kv][nb][32][head_dim/32]     E8M0 bytes, column d
 *                                                     at [d % 32][d / 32]
 * The scales start at byte offset efq_vhat_scale_offset(s).  Within the 16
 * code bytes the 32 keys are stored in the order the FP4 matrix core reads
 * them: key t of the block sits in nibble e(t) = 8*(2*((t>>2)&1) + (t>>4))
 * + 2*(t&3) + ((t>>3)&1) (byte e/2, low nibble for even e).
 * ------------------------------------------------------------------------- */
size_t efq_vhat_bytes(const efq_shape *s);
size_t efq_vhat_scale_offset(const efq_shape *s);

/* V -> V~ (MXFP4).  v: bf16 [batch][seq_k][heads_kv][head_dim]; vhat: a
 * device buffer of efq_vhat_bytes(s) bytes.  seq_q and heads_q are ignored. */
int efq_quant_v_mxfp4(const void *v, const efq_shape *s, void *vhat, size_t vhat_bytes,
                      efq_stream_t stream);

/* Attention forward on a pre-quantised V~ (output of efq_quant_v_mxfp4 for
 * the same shape).  kind: enum efq_pgen_kind; p: (tau, h) for EFQ and LUT,
 * ignored otherwise.  scale: the softmax scale, typically 1/sqrt(head_dim). */
int efq_attn_fwd_vhat(const void *q, const void *k, const void *vhat, size_t vhat_bytes,
                      float scale, int causal, int kind, efq_params p, float *out,
                      const efq_shape *s, efq_stream_t stream);

/* Both steps with a caller-owned workspace of at least
 * efq_attn_workspace_bytes(s) bytes (ws may be NULL when ws_bytes == 0: then
 * the library takes a stream-ordered allocation). */
size_t efq_attn_workspace_bytes(const efq_shape *s);
int efq_attn_fwd_ex(const void *q, const void *k, const void *v, float scale, int causal,
                    int kind, efq_params p, float *out, const efq_shape *s, void *ws,
                    size_t ws_bytes, efq_stream_t stream);

/* efq_attn_fwd_ex without any allocation, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc).  V~ goes into a scratch array the library
 * holds in device memory, EFQ_NOALLOC_SCRATCH_BYTES per GPU, for the life of
 * the process; the caller passes inputs and output as in efq_attn_fwd_ex.
 * Shapes whose V~ (efq_vhat_bytes) exceeds that size are rejected with
 * EFQ_EWORKSPACE and nothing is enqueued.  The first call on a device, with
 * that device current, looks up the array's address on the device; no call
 * allocates or frees memory.  Every call on one GPU uses the same array, so
 * calls that overlap in time on one GPU (different streams, or different
 * host threads) race and must be ordered by the caller. */
#define EFQ_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
int efq_attn_fwd_noalloc(const void *q, const void *k, const void *v, float scale, int causal,
                         int kind, efq_params p, float *out, const efq_shape *s,
                         efq_stream_t stream);

/* The two entry points of the method: EFQ-Softmax with the Mean operating
 * point, and the exp-then-quantize MXFP4 baseline. */
int efq_attn_fwd(const void *q, const void *k, const void *v, float scale, int causal,
                 float *out, const efq_shape *s, efq_stream_t stream);
int efq_attn_fwd_expq(const void *q, const void *k, const void *v, float scale, int causal,
                      float *out, const efq_shape *s, efq_stream_t stream);

/* ---------------------------------------------------------------------------
 * Low-bit Q K^T.  The paper places EFQ inside low-bit attention, whose Q K^T
 * also runs on FP8 matrix engines (Sec. I).  Here Q and K are MXFP8 under
 * the OCP microscaling rule: per row and 32 consecutive head-dim elements
 * an E8M0 exponent k = floor(log2 amax) - 8 (8 = the largest E4M3 exponent;
 * k = -127 for a block whose amax is 0 or below the normal bf16 range),
 * elements E4M3 (OCP E4M3FN, bias 7) of |x| 2^-k rounded to nearest even
 * and saturating at 448, sign bit = sign of the bf16 input.  S = Q K^T then
 * runs on the block-scaled FP8 matrix core; everything after the scores is
 * as in efq_attn_fwd_vhat.
 *
 * Q^ layout, with sq_pad = 64 * ceil(seq_q / 64) (rows past seq_q are zero):
 *   codes  [batch][heads_q][sq_pad][head_dim]      E4M3 bytes
 *   scales [batch][heads_q][sq_pad][head_dim/32]   E8M0 bytes, starting at
 *                                                  efq_qhat_scale_offset(s)
 * K^ likewise with heads_kv, seq_k and efq_khat_scale_offset(s).
 * ------------------------------------------------------------------------- */
size_t efq_qhat_bytes(const efq_shape *s);
size_t efq_qhat_scale_offset(const efq_shape *s);
size_t efq_khat_bytes(const efq_shape *s);
size_t efq_khat_scale_offset(const efq_shape *s);

/* Q, K (bf16 BSHD, device) -> Q^ and K^ (device buffers of at least
 * efq_qhat_bytes(s) and efq_khat_bytes(s) bytes). */
int efq_quant_qk_mxfp8(const void *q, const void *k, const efq_shape *s, void *qhat,
                       size_t qhat_bytes, void *khat, size_t khat_bytes, efq_stream_t stream);

/* Attention forward on Q^, K^ (efq_quant_qk_mxfp8) and V~ (efq_quant_v_mxfp4)
 * of the same shape; kind, p, scale and out as in efq_attn_fwd_vhat. */
int efq_attn_fwd_qk8(const void *qhat, size_t qhat_bytes, const void *khat, size_t khat_bytes,
                     const void *vhat, size_t vhat_bytes, float scale, int causal, int kind,
                     efq_params p, float *out, const efq_shape *s, efq_stream_t stream);

/* efq_attn_fwd_qk8 recording the probability stage, as efq_attn_fwd_dump. */
int efq_attn_fwd_qk8_dump(const void *qhat, size_t qhat_bytes, const void *khat,
                          size_t khat_bytes, const void *vhat, size_t vhat_bytes, float scale,
                          int causal, int kind, efq_params p, float *out, const efq_shape *s,
                          uint8_t *p_codes, uint8_t *p_e8m0, float *row_m, float *row_l,
                          efq_stream_t stream);

/* All three quantisers and the attention with one workspace of at least
 * efq_attn_lowbit_workspace_bytes(s) bytes, 256-byte aligned (Q^, K^ and V~
 * at 256-byte boundaries in that order); ws may be NULL with ws_bytes == 0
 * (one stream-ordered allocation, released on the same stream). */
size_t efq_attn_lowbit_workspace_bytes(const efq_shape *s);
int efq_attn_fwd_lowbit_ex(const void *q, const void *k, const void *v, float scale, int causal,
                           int kind, efq_params p, float *out, const efq_shape *s, void *ws,
                           size_t ws_bytes, efq_stream_t stream);

/* ---------------------------------------------------------------------------
 * Offline selection of (tau, h), Algorithm 3 and Sec. III-C: for every
 * candidate pair (taus[i], hs[j]), i outer and j inner, run the EFQ attention
 * forward on the calibration inputs and compute
 *   rho(tau, h) = ||O~(tau, h) - O_ref||_F / ||O_ref||_F
 * (sums of squares in fp64, reduced in a fixed order).  *best receives the
 * first pair with the smallest rho (a later pair replaces it only when
 * strictly smaller), rho (host, may be NULL) the [ntau][nh] objective grid.
 *   q, k, v   device, as for efq_attn_fwd (the calibration inputs)
 *   o_ref     device fp32 [batch][seq_q][heads_q][head_dim]: the reference
 *             output (e.g. exact softmax attention); it must not be all zero
 *   taus, hs  host arrays of ntau and nh candidates (finite, h > 0),
 *             at most 65536 pairs
 *   ws        device workspace of efq_calibrate_workspace_bytes(s, ntau*nh)
 *             bytes, 256-byte aligned, or NULL with ws_bytes == 0 (then one
 *             stream-ordered allocation is taken and released)
 * Unlike the other entry points this call waits for `stream` to finish
 * (the selection needs the objective values on the host).
 * ------------------------------------------------------------------------- */
size_t efq_calibrate_workspace_bytes(const efq_shape *s, int ncand);
int efq_calibrate(const void *q, const void *k, const void *v, float scale, int causal,
                  const float *o_ref, const efq_shape *s, const float *taus, int ntau,
                  const float *hs, int nh, double *rho, efq_params *best, void *ws,
                  size_t ws_bytes, efq_stream_t stream);

/* ---------------------------------------------------------------------------
 * Diagnostics.
 * ------------------------------------------------------------------------- */

/* The P-gen unit of Sec. III-D on its own: shifted scores x (device, fp32,
 * rows x cols row-major, every value <= 0 or -inf for a masked key) ->
 * codes (device, rows x ceil(cols/2) bytes, key 2j in the low nibble of byte
 * j) and one E8M0 byte per row and 32-column block (device, rows x
 * ceil(cols/32)).  A partial last block is padded with masked keys.  Runs
 * the same register-level code path as the fused kernel (scale 1, running
 * maximum 0).  kind: EFQ, EXPQ, EXPQ6 or LUT. */
int efq_pgen(const float *x, int rows, int cols, int kind, efq_params p, uint8_t *codes,
             uint8_t *e8m0, efq_stream_t stream);

/* Attention forward that also records what the probability stage produced
 * (small shapes): p_codes [batch][heads_q][seq_q][nblk*16] (nblk =
 * ceil(seq_k/32), key 2j in the low nibble of byte j), p_e8m0
 * [batch][heads_q][seq_q][nblk], and per row the final running maximum
 * row_m (score units) and denominator row_l.  Blocks the kernel never
 * reaches (past the causal limit) read as codes 0 and E8M0 0x00.  All four
 * buffers are device memory owned by the caller. */
int efq_attn_fwd_dump(const void *q, const void *k, const void *vhat, size_t vhat_bytes,
                      float scale, int causal, int kind, efq_params p, float *out,
                      const efq_shape *s, uint8_t *p_codes, uint8_t *p_e8m0, float *row_m,
                      float *row_l, efq_stream_t stream);

/* Register-resident P-gen throughput probe: each of `waves` wavefronts
 * (64 lanes, 32 query rows x 64 keys per tile) runs the probability stage of
 * the fused kernel `iters` times on synthetic scores and folds the result
 * into checksum[wave] (device, `waves` uint32).  kind: EFQ, EXPQ, EXPQ6 or LUT. */
int efq_pgen_bench(int kind, efq_params p, int waves, int iters, uint32_t *checksum,
                   efq_stream_t stream);

/* Shader-clock probe (diagnostic; the roofline peaks are quoted at the
 * 2.4 GHz peak clock, and the clock the matrix cores actually run at under
 * load sets what a kernel can reach).  `blocks` workgroups of four waves
 * each stream bf16 32x32x16 MFMAs, with operands that change every
 * instruction, for iters x 16 MFMAs per wave (launches of a few
 * milliseconds back to back give the clock the power limit holds); out
 * (device, 2 x blocks uint64, caller-owned) receives per workgroup the
 * s_memtime ticks (shader clock) and the s_memrealtime ticks (100 MHz) of
 * the loop, so the clock in GHz is 0.1 x out[2i] / out[2i + 1].  blocks in
 * [1, 65535], iters in [1, 2^20]; EFQ_EINVAL otherwise, before any HIP
 * call. */
int efq_clock_probe(int blocks, int iters, uint64_t *out, efq_stream_t stream);

const char *efq_strerror(int status);

/* ABI version of this header. */
#define EFQ_ABI_VERSION 1
int efq_abi_version(void);

#ifdef __cplusplus
}
#endif
#endif /* EFQ_ATTN_H */
