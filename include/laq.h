/*
 * laq.h -- C ABI of the MI355X (gfx950) W3G128 / W4G128 weight-only quantized
 * linear library for LAQuant (arXiv 2605.08755).
 *
 * LAQuant's deployed model is a standard weight-only quantized model: integer
 * codes plus a scale and a zero point per group of 128 consecutive weights of
 * a row, with no online rotation (Sec. 3, "Runtime-Overhead-Free
 * Quantization"; Sec. 5 efficiency results).  This library provides the two
 * operations on that model's decode hot path, as hand-written HIP kernels:
 *
 *   laq_quantize_w3g128 -- Eq. 1 (Sec. 2): q = clip(round(w/s) + z, 0, 7)
 *                          with round-to-nearest min-max s, z per 128-group,
 *                          packed 32 codes per three 32-bit words (App. H).
 *   laq_pack_w3g128     -- Eq. 1 with caller-supplied s, z (for instance the
 *                          scale and zero point LAQuant's QAT learned),
 *                          packed the same way.
 *   laq_linear_w3g128   -- y = x * w_hat^T with w_hat = s * (q - z) (Eq. 1),
 *                          the fused dequantize GEMV / skinny GEMM of decode
 *                          (App. H describes the paper's INT3 GEMV).
 *
 * plus the W4G128 (4-bit, 8 codes per word) siblings used for bit-width
 * comparison (Table 3 reports W4G128 and W3G128 decoding).
 *
 * Conventions for every entry point
 * ---------------------------------
 *  - Tensor pointers are DEVICE pointers into memory the caller owns and
 *    keeps alive until the stream work completes.  The library never
 *    allocates, frees or synchronizes inside these calls (scratch memory,
 *    where a call can use it, is a caller-provided workspace).
 *  - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *    Work is enqueued asynchronously; results are valid once the caller
 *    synchronizes with the stream.
 *  - Arguments are validated on the host before anything is enqueued.  On
 *    any error nothing is enqueued and outputs are left untouched; the call
 *    returns a laq_status and laq_last_error() gives a message.
 *  - Outputs must not alias inputs.  Weights and activations must be finite.
 *  - Shapes: N >= 1 output features, K >= 128 input features with
 *    K % 128 == 0, 1 <= M <= 16 activation rows; N*K < 2^40.
 *  - Results are deterministic: the same inputs give bitwise-identical
 *    outputs, call after call.  Calls are thread-safe and may run
 *    concurrently on different streams.
 *
 * Data layout (G = K/128 groups per row, C = K/32 chunks per row)
 * --------------------------------------------------------------
 *  w        fp16 [N][K], row-major (PyTorch Linear weight, (out, in)).
 *  x        fp16 [M][K], row-major.
 *  y        fp16 [M][N], row-major.
 *  scales   fp16 [N][G]   -- s of group g of row n at scales[n*G + g].
 *  zeros    uint8 [N][G]  -- z (0..2^b-1) of group g of row n.
 *  qweight  W3: uint32 [N][3][C]; W4: uint32 [N][4][C].
 *    Chunk c of row n covers k = 32c .. 32c+31 and is stored in the words
 *    P_p = qweight[(n*B + p)*C + c] for planes p = 0..B-1 (B = 3 or 4), so
 *    32 codes occupy exactly three (W3) or four (W4) 32-bit words.
 *    W3, code i of the chunk (bits of the code LSB first):
 *      i < 30: plane i/10; with r = i%10, bits [16*(r%2) + OFF[r/2], +3)
 *              where OFF = {0, 3, 6, 10, 13};
 *      i = 30: code bit j is bit 9 of plane j (j = 0, 1, 2);
 *      i = 31: code bit j is bit 25 of plane j.
 *    W4, code i of the chunk: plane i/8, bits [16*(i%2) + 4*((i%8)/2), +4).
 *    Each code pair (2t, 2t+1) thus sits at the same offset in the low and
 *    high 16-bit halves of a word, inside the fp16 mantissa field, which is
 *    what lets the GEMV turn one masked word into two fp16 operands.
 *
 * Alignment: w, x and qweight 16-byte aligned; scales and y 2-byte aligned.
 */
#ifndef LAQ_H
#define LAQ_H

#include <stdint.h>
#include <stddef.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t laq_status;

#define LAQ_OK                0
#define LAQ_ERR_NULL_POINTER  1  /* a required pointer is NULL               */
#define LAQ_ERR_BAD_SHAPE     2  /* N < 1, K < 128, K % 128 != 0, too large  */
#define LAQ_ERR_BAD_M         3  /* M outside 1..16                          */
#define LAQ_ERR_MISALIGNED    4  /* a pointer violates its alignment         */
#define LAQ_ERR_HIP           5  /* the HIP runtime reported an error        */

#define LAQ_ABI_VERSION 1
#define LAQ_GROUP 128
#define LAQ_MAX_M 16
#define LAQ_MAX_GROUP 8

/* ABI version of the loaded library (LAQ_ABI_VERSION it was built with). */
int32_t laq_abi_version(void);

/* Static description of a status code. */
const char *laq_status_string(laq_status status);

/* Detail message of the last failing call on this host thread ("" if none). */
const char *laq_last_error(void);

/*
 * laq_profile_next_launch -- measurement hook, not needed for normal use.
 * The next laq_quantize_* / laq_linear_* call made on this host thread
 * records `start_event` when its kernel starts executing and `stop_event`
 * when it ends (hipEvent_t handles created by the caller, passed as void*;
 * either may be NULL), so hipEventElapsedTime gives the kernel's own
 * duration without launch gaps.  The hook is then cleared.  A call that
 * fails validation also clears it.  Always returns LAQ_OK.
 */
laq_status laq_profile_next_launch(void *start_event, void *stop_event);

/*
 * laq_quantize_w3g128 -- Eq. 1 (Sec. 2) with round-to-nearest min-max
 * parameters, per group of 128 consecutive weights of a row.
 *
 * For row n and group g, in IEEE fp32 with round-half-to-even:
 *   lo = min(0, min w), hi = max(0, max w)
 *   s16 = fp16(fl32(hi - lo) / 7); s16 = 2^-24 if it rounds to zero
 *   z   = clamp(rint(-lo / s16), 0, 7)
 *   q   = clamp(rint(w / s16) + z, 0, 7)          (true division)
 * and writes q packed as described above, s16 to scales and z to zeros.
 *
 *   w        [in]  fp16 [N][K]
 *   qweight  [out] uint32 [N][3][K/32]   (N*K*3/8 bytes)
 *   scales   [out] fp16 [N][K/128]
 *   zeros    [out] uint8 [N][K/128]
 */
laq_status laq_quantize_w3g128(const void *w, int64_t N, int64_t K,
                               uint32_t *qweight, void *scales, uint8_t *zeros,
                               void *stream);

/*
 * laq_pack_w3g128 -- Eq. 1 (Sec. 2) with caller-supplied parameters: the
 * scale and zero point of every group are inputs (LAQuant learns them by
 * QAT, Sec. 3; the deployed model is these codes plus those parameters).
 *
 * For row n, group g and every weight w of the group, in IEEE fp32 with
 * round-half-to-even:
 *   s = scales[n][g] (fp16, must be finite and > 0), z = zeros[n][g] (0..7)
 *   q = clip(rint(w / s) + z, 0, 7)          (true division; the clip is on
 *                                             the real value)
 * and writes q packed exactly as laq_quantize_w3g128 does.  Fed the scales
 * and zeros that laq_quantize_w3g128 wrote, it reproduces that call's
 * qweight bit for bit.  scales and zeros are only read.
 *
 *   w        [in]  fp16 [N][K]
 *   scales   [in]  fp16 [N][K/128]
 *   zeros    [in]  uint8 [N][K/128]
 *   qweight  [out] uint32 [N][3][K/32]
 */
laq_status laq_pack_w3g128(const void *w, const void *scales, const uint8_t *zeros,
                           int64_t N, int64_t K, uint32_t *qweight, void *stream);

/*
 * laq_linear_w3g128 -- y[m][n] = sum_k x[m][k] * s[n][g] * (q[n][k] - z[n][g]),
 * g = k/128: the dequantize-fused GEMV (M = 1) / skinny GEMM (M <= 16) of
 * decoding.  fp16 inputs, fp32 accumulation, one fp16 round-to-nearest-even
 * rounding of each output.
 *
 *   x        [in]  fp16 [M][K]
 *   qweight, scales, zeros [in] as written by laq_quantize_w3g128 (or by any
 *            producer of the same layout, e.g. trained QAT parameters)
 *   y        [out] fp16 [M][N]
 */
laq_status laq_linear_w3g128(const void *x, const uint32_t *qweight,
                             const void *scales, const uint8_t *zeros,
                             void *y, int64_t M, int64_t N, int64_t K,
                             void *stream);

/*
 * laq_linear_workspace_bytes -- device workspace (bytes) with which
 * laq_linear_ws_w3g128 / laq_linear_ws_w4g128 split K across workgroups for
 * an (M, N, K) call: the reduction along K of Eq. 1's dot products, which
 * App. H's GEMV spreads over a 2-D grid of thread blocks, here deterministic
 * (fp32 partial sums per K range, added in a fixed order by a second kernel).
 * It applies on the matrix-core path (M >= 2) to rows of at least 40 quads
 * of four groups (K > 19968) and fewer than 1024 tiles of 16 rows
 * (N <= 16368): there, four tiles per workgroup share each activation slab
 * and the K ranges give every compute unit work, which outweighs the second
 * kernel (measured on MI355X: Qwen3-32B down projection, N = 5120,
 * K = 25600, M = 16: 33.2 -> 31.3 us; shorter rows measured slower split).  Returns 0 when the call
 * never splits K (then the _ws entry point is the plain one), otherwise an
 * upper bound of what the call uses.  Depends on the shape only (not on the
 * bit width); an invalid shape gives 0.
 */
int64_t laq_linear_workspace_bytes(int64_t M, int64_t N, int64_t K);

/*
 * laq_linear_ws_w3g128 -- laq_linear_w3g128 with a caller-provided workspace.
 *
 *   workspace        [scratch] device memory, 16-byte aligned, any contents;
 *                    the call writes and reads it (fp32 partial sums).  It
 *                    must overlap no other argument and serve no other call
 *                    in flight (one workspace per stream).  May be NULL when
 *                    workspace_bytes is 0.
 *   workspace_bytes  [in] its size.  With workspace_bytes >=
 *                    laq_linear_workspace_bytes(M, N, K) > 0 the call splits
 *                    K; otherwise it is laq_linear_w3g128.
 *
 * Results: within the linear tolerance of laq_linear_w3g128 (the fp32 sums
 * are added in another order), bitwise-identical from call to call for the
 * same shape.  The call enqueues two kernels when it splits K.
 */
laq_status laq_linear_ws_w3g128(const void *x, const uint32_t *qweight,
                                const void *scales, const uint8_t *zeros,
                                void *y, int64_t M, int64_t N, int64_t K,
                                void *workspace, int64_t workspace_bytes,
                                void *stream);

/*
 * laq_linear_noalloc_w3g128 -- for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid allocation): laq_linear_ws_w3g128 with the split-K partial sums in a
 * scratch array the library itself holds on each GPU, instead of a caller's
 * workspace.  The call allocates nothing.
 *
 *   Arguments, layouts and results as for laq_linear_w3g128; the results
 *   equal laq_linear_ws_w3g128's with a large enough workspace, bit for bit.
 *   Scratch: LAQ_NOALLOC_SCRATCH_BYTES (8 MiB) per GPU, held from the first
 *   call on that GPU until the process ends.  A shape whose partial sums
 *   (laq_linear_workspace_bytes(M, N, K)) exceed it is rejected with
 *   LAQ_ERR_BAD_SHAPE before anything is enqueued.  Every call on a GPU
 *   shares that GPU's array: calls that may overlap in time on one GPU (on
 *   different streams, or from several host threads) race on it and must be
 *   ordered by the caller; the partial sums are fully written before they
 *   are read, so nothing needs clearing between calls.
 */
#define LAQ_NOALLOC_SCRATCH_BYTES (8 << 20)
laq_status laq_linear_noalloc_w3g128(const void *x, const uint32_t *qweight,
                                     const void *scales, const uint8_t *zeros,
                                     void *y, int64_t M, int64_t N, int64_t K,
                                     void *stream);

/*
 * laq_linear_swiglu_w3g128 -- the gate|up projection of a SwiGLU MLP block
 * with SiLU-and-multiply in its output stage (the decode step's MLP input,
 * one launch instead of a linear and a separate elementwise kernel).  The
 * weight rows come in pairs: row 2j is gate row j and row 2j + 1 is up row j
 * (quantized as any other rows).  With a = sum_k x[m][k] s[2j][g] (q - z) and
 * b the same sum over row 2j + 1, both in fp32,
 *   y[m][j] = fp16(a / (1 + exp(-a)) * b),   j < N / 2
 * rounded once (a and b are not rounded to fp16 first).
 *
 *   x        [in]  fp16 [M][K], 1 <= M <= 4
 *   qweight, scales, zeros [in] as for laq_linear_w3g128, N rows, N even
 *   y        [out] fp16 [M][N/2]
 *   K        K <= 16384 / M' with M' = M rounded up to 1, 2 or 4 (the
 *            activation tile stays in LDS); larger shapes: LAQ_ERR_BAD_SHAPE.
 */
laq_status laq_linear_swiglu_w3g128(const void *x, const uint32_t *qweight,
                                    const void *scales, const uint8_t *zeros,
                                    void *y, int64_t M, int64_t N, int64_t K,
                                    void *stream);

/*
 * laq_linear_group_w3g128 -- several independent laq_linear_w3g128 calls
 * (1 <= count <= LAQ_MAX_GROUP) with the same M, issued as one kernel launch:
 * for instance the q, k and v projections of a decoder layer, which read the
 * same activations, without concatenating their weights.  A decode step's
 * stages depend on each other through attention and normalization, so only
 * calls that share a stage can be grouped; one launch instead of one per
 * call is what the grouping saves (a dependent launch costs about 1.6 us on
 * MI355X).
 *
 *   calls  [in]  host array of `count` descriptors; each is validated as the
 *                corresponding laq_linear_w3g128 call would be.  The calls
 *                must be independent: no call's y may overlap any call's x,
 *                weights or y.
 *   M      [in]  activation rows of every call, 1..16.
 *
 * Results: each y equals that call's laq_linear_w3g128 result within the
 * linear tolerance; on the one-row VALU path (M <= 2, and M <= 4 with rows of
 * at most 3072) bit for bit.  One activation row longer than the LDS holds
 * (K > ~29000) makes the group one launch per call, with the same results.
 */
typedef struct laq_linear_call {
    const void *x;            /* fp16 [M][K] */
    const uint32_t *qweight;  /* [N][bits][K/32] */
    const void *scales;       /* fp16 [N][K/128] */
    const uint8_t *zeros;     /* uint8 [N][K/128] */
    void *y;                  /* fp16 [M][N] (output) */
    int64_t N;
    int64_t K;
} laq_linear_call;

laq_status laq_linear_group_w3g128(const laq_linear_call *calls, int32_t count, int64_t M,
                                   void *stream);

/* W4G128 siblings: same contracts with 4-bit codes (0..15), s = (hi-lo)/15,
 * zero points 0..15, qweight uint32 [N][4][K/32] (N*K/2 bytes). */
laq_status laq_quantize_w4g128(const void *w, int64_t N, int64_t K,
                               uint32_t *qweight, void *scales, uint8_t *zeros,
                               void *stream);

laq_status laq_pack_w4g128(const void *w, const void *scales, const uint8_t *zeros,
                           int64_t N, int64_t K, uint32_t *qweight, void *stream);

laq_status laq_linear_group_w4g128(const laq_linear_call *calls, int32_t count, int64_t M,
                                   void *stream);

laq_status laq_linear_w4g128(const void *x, const uint32_t *qweight,
                             const void *scales, const uint8_t *zeros,
                             void *y, int64_t M, int64_t N, int64_t K,
                             void *stream);

laq_status laq_linear_ws_w4g128(const void *x, const uint32_t *qweight,
                                const void *scales, const uint8_t *zeros,
                                void *y, int64_t M, int64_t N, int64_t K,
                                void *workspace, int64_t workspace_bytes,
                                void *stream);

laq_status laq_linear_swiglu_w4g128(const void *x, const uint32_t *qweight,
                                    const void *scales, const uint8_t *zeros,
                                    void *y, int64_t M, int64_t N, int64_t K,
                                    void *stream);

/* ------------------------------------------------------------------------
 * Decode-step operations around the linears of a decoder layer (the model
 * the paper quantizes and times, Sec. 5, Table 3), for one decode token.
 * fp16 arrays are IEEE binary16; arithmetic is fp32 with fixed reduction
 * orders (deterministic).  Head dimension 128.  Same conventions as above:
 * host-side validation, nothing enqueued on error, asynchronous on `stream`,
 * no allocation; outputs must not alias inputs unless stated.
 * ------------------------------------------------------------------------ */

/* laq_add_rmsnorm_linear_w3g128 -- laq_add_rmsnorm_f16 for one token (M = 1,
 * D = K) followed by laq_linear_w3g128 on its output, in one kernel: every
 * block of the linear forms
 *   r = residual + delta;  x = fp16(r / sqrt(mean(r^2) + eps) * norm_weight)
 * itself while it stages its activation row (the decode step's norms before
 * the attention and before the MLP feed a linear; Sec. 5, Table 3 setting),
 * and y = x w_hat^T as laq_linear_w3g128 (Eq. 1 dequantization, App. H
 * format).  The normalized row is not written.
 *   residual      [in] fp32 [K], 16-byte aligned.
 *   delta         [in] fp16 [K], 16-byte aligned, or NULL (then r = residual).
 *   norm_weight   [in] fp16 [K], 16-byte aligned.
 *   residual_out  [out] fp32 [K], 16-byte aligned, receives r; or NULL.  Must
 *                 not overlap residual (the blocks read residual while one of
 *                 them writes r).
 *   qweight, scales, zeros, y, N  as laq_linear_w3g128 with M = 1.
 * Results: y within the linear's tolerance of the two-call sequence (the
 * sum of squares is added in another order; x can differ by one fp16 ulp),
 * r bitwise equal to laq_add_rmsnorm_f16's residual; deterministic.
 * Errors: NULL_POINTER (residual, norm_weight, qweight, scales, zeros, y);
 * BAD_SHAPE (N < 1, K not a multiple of 128, K > 8192, eps < 0 or not finite,
 * residual_out overlapping residual); MISALIGNED. */
laq_status laq_add_rmsnorm_linear_w3g128(const float *residual, const void *delta, const void *norm_weight,
                                         float eps, float *residual_out, const uint32_t *qweight,
                                         const void *scales, const uint8_t *zeros, void *y, int64_t N,
                                         int64_t K, void *stream);

/* laq_add_rmsnorm_linear_swiglu_w3g128 -- the same prologue followed by
 * laq_linear_swiglu_w3g128 (gate and up rows interleaved, N even, y fp16
 * [N/2] = silu(gate) * up). */
laq_status laq_add_rmsnorm_linear_swiglu_w3g128(const float *residual, const void *delta,
                                                const void *norm_weight, float eps, float *residual_out,
                                                const uint32_t *qweight, const void *scales,
                                                const uint8_t *zeros, void *y, int64_t N, int64_t K,
                                                void *stream);

/* W4G128 siblings of the two calls above (qweight as laq_linear_w4g128). */
laq_status laq_add_rmsnorm_linear_w4g128(const float *residual, const void *delta, const void *norm_weight,
                                         float eps, float *residual_out, const uint32_t *qweight,
                                         const void *scales, const uint8_t *zeros, void *y, int64_t N,
                                         int64_t K, void *stream);

laq_status laq_add_rmsnorm_linear_swiglu_w4g128(const float *residual, const void *delta,
                                                const void *norm_weight, float eps, float *residual_out,
                                                const uint32_t *qweight, const void *scales,
                                                const uint8_t *zeros, void *y, int64_t N, int64_t K,
                                                void *stream);

/* laq_linear_residual_w3g128 -- a batch-1 linear that also updates the
 * residual stream: y = x w_hat^T exactly as laq_linear_w3g128 with M = 1
 * (Eq. 1 dequantization, App. H format; bit for bit the same y), and
 *   residual_out[n] = residual_in[n] + y[n]      (fp32 + the fp16 output)
 * for every output row n (the decode step's o and down projections, whose
 * outputs the residual stream adds; Sec. 5, Table 3 setting).  The next
 * norm then reads the new residual with no delta (laq_add_rmsnorm_linear_*
 * with delta NULL).
 *   x, qweight, scales, zeros, N, K  as laq_linear_w3g128 with M = 1.
 *   y             [out] fp16 [N], 2-byte aligned, or NULL: then only
 *                 residual_out is written (a decode step whose next norm
 *                 reads the residual alone needs no y).
 *   residual_in   [in] fp32 [N], 4-byte aligned.
 *   residual_out  [out] fp32 [N], 4-byte aligned; may be residual_in itself
 *                 (in place), otherwise must not overlap it.
 * Errors: NULL_POINTER; BAD_SHAPE (shape rules of laq_linear_w3g128, K below
 * 2048, rows too long for one activation tile in LDS (K above about 28000),
 * partial overlap of the residuals); MISALIGNED. */
laq_status laq_linear_residual_w3g128(const void *x, const uint32_t *qweight, const void *scales,
                                      const uint8_t *zeros, void *y, const float *residual_in,
                                      float *residual_out, int64_t N, int64_t K, void *stream);

/* W4G128 sibling (qweight as laq_linear_w4g128). */
laq_status laq_linear_residual_w4g128(const void *x, const uint32_t *qweight, const void *scales,
                                      const uint8_t *zeros, void *y, const float *residual_in,
                                      float *residual_out, int64_t N, int64_t K, void *stream);

/* laq_mlp_workspace_bytes -- device workspace (bytes) that
 * laq_add_rmsnorm_mlp_w3g128 needs for hidden size D and MLP width I
 * (fp32 partial sums per 128 intermediates, fp32 team sums, counters);
 * 0 when the shape is not supported. */
int64_t laq_mlp_workspace_bytes(int64_t D, int64_t I);

/* laq_add_rmsnorm_mlp_w3g128 -- the SwiGLU MLP block of one token in one
 * launch (the decode step's post-attention half of a decoder layer; Sec. 5,
 * Table 3 setting; every weight dequantized by Eq. 1 in the App. H format):
 *   r = residual + delta;  x = fp16(r / sqrt(mean(r^2) + eps) * norm_weight)
 *   h = fp16(silu(x gate^T) * (x up^T))          (fp16 [I])
 *   y = fp16(h down^T)                           (fp16 [D])
 * with the norm as laq_add_rmsnorm_linear_w3g128 and h as
 * laq_add_rmsnorm_linear_swiglu_w3g128.  The down product is split over I in
 * slices of 128 (one workgroup each); the slices' fp32 partial sums are added
 * in a fixed order by the last workgroups to finish, so y is deterministic.
 *   residual, delta, norm_weight, eps, residual_out  as for
 *                 laq_add_rmsnorm_linear_w3g128 (K = D).
 *   gu_qweight, gu_scales, gu_zeros  [in] gate|up weights, 2I rows of D
 *                 (gate row j, up row j interleaved) as for
 *                 laq_linear_swiglu_w3g128.
 *   down_qweight, down_scales, down_zeros  [in] down weights, D rows of I.
 *   y             [out] fp16 [D].
 *   workspace     [scratch] device memory, 16-byte aligned, at least
 *                 laq_mlp_workspace_bytes(D, I) bytes, filled with zeros once
 *                 before its first use (its counters; each call leaves them
 *                 zero again); calls in flight need separate workspaces.
 * Results: y within the linear tolerance of the three-call sequence
 * laq_add_rmsnorm_linear_swiglu_w3g128 + laq_linear_w3g128 (h can differ by
 * one fp16 ulp where x does, and the fp32 sums are added in another order);
 * r bitwise equal to laq_add_rmsnorm_f16's.
 * Errors: NULL_POINTER; BAD_SHAPE (D or I not a positive multiple of 128,
 * D > 2560, I > 2^20, eps < 0 or not finite, residual_out overlapping
 * residual, workspace too small); MISALIGNED. */
laq_status laq_add_rmsnorm_mlp_w3g128(const float *residual, const void *delta, const void *norm_weight,
                                      float eps, float *residual_out, const uint32_t *gu_qweight,
                                      const void *gu_scales, const uint8_t *gu_zeros,
                                      const uint32_t *down_qweight, const void *down_scales,
                                      const uint8_t *down_zeros, void *y, int64_t D, int64_t I,
                                      void *workspace, int64_t workspace_bytes, void *stream);

/* laq_add_rmsnorm_f16 -- residual update and RMSNorm, row by row:
 *   r = residual + delta;  y = fp16(r / sqrt(mean(r^2) + eps) * weight)
 *   residual  [in/out] fp32 [M][D]; receives r (may be read by later calls).
 *   delta     [in] fp16 [M][D], or NULL (then r = residual).
 *   weight    [in] fp16 [D].   y [out] fp16 [M][D].
 * Errors: NULL_POINTER; BAD_SHAPE (M < 1, D < 1, D > 2^20, eps < 0 or not
 * finite); MISALIGNED (residual 4-byte, fp16 arrays 2-byte). */
laq_status laq_add_rmsnorm_f16(float *residual, const void *delta, const void *weight, void *y,
                               int64_t M, int64_t D, float eps, void *stream);

/* laq_qk_norm_rope_f16 -- one token's fused q|k|v projection output
 * qkv fp16 [(Hq + 2*Hkv) * 128] (q heads, then k heads, then v heads):
 * every q and k head is RMS-normalized over its 128 values with its own
 * weight vector (q_norm_weight / k_norm_weight, fp16 [128], eps as above),
 * then rotated: pair (x_i, x_{i+64}), i < 64, becomes
 * (x_i c_i - x_{i+64} s_i, x_{i+64} c_i + x_i s_i) with c_i, s_i read from
 * row pos of cos_sin (fp32 [S_max][128]: the 64 cosines of pos * theta_i,
 * then the 64 sines; the caller chooses the frequencies theta_i).  q heads go
 * to q_out fp16 [Hq][128]; k and v heads to row pos of k_cache / v_cache,
 * fp16 [Hkv][S_max][128] each (16-byte aligned).
 * Errors: NULL_POINTER; BAD_SHAPE (head_dim != 128, Hq not Hkv times 1, 2, 4
 * or 8, Hq > 4096, pos outside 0..S_max-1, S_max > 2^21, bad eps);
 * MISALIGNED. */
laq_status laq_qk_norm_rope_f16(const void *qkv, const void *q_norm_weight, const void *k_norm_weight,
                                const float *cos_sin, int64_t pos, int64_t Hq, int64_t Hkv,
                                int64_t head_dim, float eps, void *q_out, void *k_cache, void *v_cache,
                                int64_t S_max, void *stream);

/* laq_decode_attention_workspace_bytes -- workspace (bytes) that
 * laq_decode_attention_f16 needs for Hq query heads over L positions
 * (fp32 partial results per block of 64 positions); 0 for invalid sizes. */
int64_t laq_decode_attention_workspace_bytes(int64_t Hq, int64_t L);

/* laq_decode_attention_f16 -- single-token attention over the first L
 * positions of the caches: query head h (q fp16 [Hq][128]) reads key/value
 * head h / (Hq / Hkv);
 *   out[h] = sum_t softmax_t(q[h] . k[t] / sqrt(128)) v[t]   (fp16 [Hq][128])
 * Two kernels: partial results per block of 64 positions into the caller's
 * workspace, then their combination in position order.
 *   workspace  [scratch] device memory, 16-byte aligned, any contents, at
 *              least laq_decode_attention_workspace_bytes(Hq, L) bytes; calls
 *              in flight need separate workspaces.
 * Errors: NULL_POINTER; BAD_SHAPE (head layout as above, L outside
 * 1..S_max, S_max > 2^21, workspace too small); MISALIGNED. */
laq_status laq_decode_attention_f16(const void *q, const void *k_cache, const void *v_cache, int64_t Hq,
                                    int64_t Hkv, int64_t head_dim, int64_t L, int64_t S_max, void *out,
                                    void *workspace, int64_t workspace_bytes, void *stream);

/* laq_decode_attention_qkv_workspace_bytes -- workspace (bytes) with which
 * laq_decode_attention_qkv_f16 runs for Hq query heads, Hkv key/value heads
 * and any pos with pos + 1 <= L (so one workspace sized for L = S_max serves a
 * whole generation); 0 for invalid sizes. */
int64_t laq_decode_attention_qkv_workspace_bytes(int64_t Hq, int64_t Hkv, int64_t L);

/* laq_decode_attention_qkv_f16 -- laq_qk_norm_rope_f16 followed by
 * laq_decode_attention_f16 over L = pos + 1 positions, in two kernels
 * instead of three: from one token's q|k|v projection output qkv (layout as
 * for laq_qk_norm_rope_f16), each q and k head is RMS-normalized with its
 * weights and rotated by row pos of cos_sin; k and v are written to row pos of
 * the caches; then
 *   out[h] = sum_{t <= pos} softmax_t(q[h] . k[t] / sqrt(128)) v[t]
 * (fp16 [Hq][128]) with q rounded to fp16 as laq_qk_norm_rope_f16 stores it.
 * The positions are split into tiles of 16, 32 or 64 (so that short contexts
 * still occupy the GPU), whose partial results go to the workspace and are
 * combined in position order.  Results: within the tolerance of the
 * two-call sequence (the tiles differ), deterministic.
 *   workspace  [scratch] device memory, 16-byte aligned, any contents, at
 *              least laq_decode_attention_qkv_workspace_bytes(Hq, Hkv, pos + 1)
 *              bytes; calls in flight need separate workspaces.
 * Errors: NULL_POINTER; BAD_SHAPE (head layout as for laq_qk_norm_rope_f16,
 * pos outside 0..S_max-1, S_max > 2^21, bad eps, workspace too small);
 * MISALIGNED. */
laq_status laq_decode_attention_qkv_f16(const void *qkv, const void *q_norm_weight, const void *k_norm_weight,
                                        const float *cos_sin, int64_t pos, int64_t Hq, int64_t Hkv,
                                        int64_t head_dim, float eps, void *k_cache, void *v_cache, int64_t S_max,
                                        void *out, void *workspace, int64_t workspace_bytes, void *stream);

/* laq_silu_mul_f16 -- y[m][i] = fp16(silu(g) * u), g = gate_up[m][i],
 * u = gate_up[m][I + i], silu(g) = g / (1 + exp(-g)): the fused gate|up
 * projection's output fp16 [M][2I] to the down projection's input
 * fp16 [M][I].
 * Errors: NULL_POINTER; BAD_SHAPE (M outside 1..65535, I outside 1..2^30);
 * MISALIGNED. */
laq_status laq_silu_mul_f16(const void *gate_up, void *y, int64_t M, int64_t I, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* LAQ_H */
