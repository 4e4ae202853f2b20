/*
 * sq.h -- C ABI of the fused low-bit linear layer of a world-action diffusion
 * Transformer (SteerQuant / Rudder, arXiv 2609.39056), for AMD MI355X (gfx950).
 *
 * The layer computes, for one linear at denoising step tau
 * (Sec. 4.3 Eq. 8 with the channel scaling of Sec. 4.2 Eq. 6):
 *
 *     Y = gamma_{tau,s}^-1 Q(gamma_{tau,s} X D^-1 ; c) Q(D W) + b
 *
 * in two kernels (Sec. 4.4): the first applies D^-1 and the stream gain while
 * quantizing and writes integer activations Q_X plus row scales
 * r_i = Delta_X / gamma_s(i); the second accumulates Q_X Q_W in int32 and
 * applies the epilogue of Eq. 10, Y_ij = cast[(fp32(C_ij) r_i) Delta_W,j + b_j].
 *
 * Conventions shared by every entry point
 * --------------------------------------
 * - Pointers named in the structs and arguments are DEVICE pointers unless
 *   stated otherwise; the structs themselves live in host memory and are
 *   read before the call returns.
 * - The caller owns every buffer.  The library allocates nothing, frees
 *   nothing, keeps no pointer after returning and never synchronizes: all work
 *   is enqueued on `stream` (a hipStream_t; NULL = the null stream).
 * - Arguments are validated on the host before anything is enqueued; a
 *   failing check returns a negative sq_status and launches nothing.  A launch
 *   failure returns SQ_ERR_HIP.  Stream ids in tok2stream are device data and
 *   are not checked: each must lie in [0, num_streams).
 * - Matrices are row-major.  X is [M, K] bf16 (K contiguous).  W is stored
 *   transposed, [N, K] (K contiguous), as packed int4.  Y is [M, N].
 * - Shapes: 1 <= M <= 2^24; K % 128 == 0 and 128 <= K <= 32768; N % 64 == 0
 *   and 64 <= N <= 2^20.
 * - Alignment: x, qx, qw, y and workspace 16 bytes; the bf16 bias 2 bytes;
 *   every other pointer 4 bytes (the kernels read the fp16 weight and group
 *   steps in pairs).
 * - Inputs must be finite; X D^-1 gamma must stay finite in fp32.
 *
 * Packed int4 layout (weights and A4 activations)
 * -----------------------------------------------
 * Codes are two's-complement nibbles.  Per row, each group of 8 consecutive
 * codes k = 8g .. 8g+7 occupies bytes 4g .. 4g+3; byte 4g+b holds code 8g+b
 * in its low nibble and code 8g+b+4 in its high nibble.
 *
 * Quantization arithmetic (both range modes; q_max = 127 for 8-bit, 7 for
 * 4-bit activations; every step is one IEEE fp32 operation, round to nearest
 * even, no contraction):
 *     x~    = fp32(x) * dinv[k]                            (Eq. 6)
 *     c     = clip[tau]  (STATIC)  |  max |x~| over the row (8-bit) or over the
 *             64-wide group (4-bit), before the gain       (DYNAMIC)
 *     Delta = c / q_max;  4-bit: Delta = fp32(fp16(Delta))  (Eq. 1)
 *     inv   = 1 / Delta, or 0 where that is infinite
 *     q     = rint(clamp((x~ * g) * inv, -q_max, q_max)),   g = gamma[tau][s(i)]
 *     8-bit: r_i = Delta / g  (fp32)                        (Sec. 4.4)
 *     4-bit: sigma_{i,a} = fp16(Delta) per 64-group; the compensation
 *            1/g is applied to the row in the GEMM epilogue (Eq. 8).
 */
#ifndef SQ_H_
#define SQ_H_

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SQ_OK = 0,
  SQ_ERR_NULL = -1,        /* a required pointer is NULL */
  SQ_ERR_SHAPE = -2,       /* a size, step index or stream count is out of range */
  SQ_ERR_ALIGN = -3,       /* a pointer is not aligned as required */
  SQ_ERR_UNSUPPORTED = -4, /* bits, group size, range mode or dtype not supported */
  SQ_ERR_WORKSPACE = -5,   /* workspace smaller than sq_workspace_bytes() */
  SQ_ERR_HIP = -6          /* a kernel launch failed */
} sq_status;

typedef enum {
  SQ_RANGE_DYNAMIC = 0, /* c = per-token (8-bit) or per-64-group (4-bit) amax of X D^-1 */
  SQ_RANGE_STATIC = 1   /* c = clip[tau], the per-step threshold of Sec. 4.3 */
} sq_range_mode;

typedef enum { SQ_OUT_F32 = 0, SQ_OUT_BF16 = 1, SQ_OUT_F16 = 2 } sq_out_dtype;

typedef enum {
  SQ_VARIANT_FUSED = 0,   /* sq_linear_w4a8 / sq_linear_w4a4 */
  SQ_VARIANT_UNFUSED = 1, /* sq_linear_unfused */
  SQ_VARIANT_GEMM = 2     /* sq_gemm_w4a8 / sq_gemm_w4a4 (optional workspace) */
} sq_variant;

/* Per-layer activation-side parameters (Sec. 4.3: gains and threshold stored
 * in a layer-step lookup table; Sec. 4.2: one channel scaling per layer). */
typedef struct sq_act_params {
  const int32_t* tok2stream; /* [M] stream id s(i) of every row, in [0, num_streams) */
  const float* gamma;        /* [num_steps][num_streams] gains, finite and > 0 */
  const float* clip;         /* [num_steps] thresholds > 0; required for STATIC, else may be NULL */
  const float* dinv;         /* [K] D^-1 (positive), or NULL for D = I */
  int32_t num_streams;       /* S >= 1 */
  int32_t num_steps;         /* T >= 1 */
  int32_t step;              /* tau, 0 <= tau < T */
  int32_t range_mode;        /* sq_range_mode */
  int32_t act_bits;          /* 8 (per-token steps) or 4 (per-64-group fp16 steps) */
} sq_act_params;

/* A prepared weight: Q(D W) with fp16 steps (Sec. 4.2, fold then pack). */
typedef struct sq_weight {
  const uint8_t* qw;        /* [N][K/2] packed int4 codes (layout above) */
  const uint16_t* w_scale;  /* [K/w_group][N] fp16 steps Delta_W, group-major: the steps of
                               one input-channel group are contiguous over output channels */
  const uint16_t* bias;     /* [N] bf16 bias b, or NULL */
  int32_t N, K;
  int32_t w_group;          /* 128, or K (one step per output channel, as in the paper) */
} sq_weight;

/* Human-readable name of a status code (static storage). */
const char* sq_status_string(int32_t status);

/* Bytes of device workspace that sq_linear_w4a8 / sq_linear_w4a4
 * (variant SQ_VARIANT_FUSED), sq_linear_unfused (SQ_VARIANT_UNFUSED) or
 * sq_gemm_w4a8 / sq_gemm_w4a4 (SQ_VARIANT_GEMM) use for this shape on the
 * current device (at least 256); 0 for invalid arguments.  Host-only.
 *
 * The GEMM part of a workspace holds fp32 partial sums: when the output tiles
 * do not fill whole rounds of the device's workgroup slots, the tiles left
 * over are split along K over the idle slots and a second kernel adds the
 * partial sums (in a fixed order: results are deterministic).  Its contents
 * need no initialization and are garbage after a call. */
size_t sq_workspace_bytes(int32_t variant, int32_t M, int32_t K, int32_t N, int32_t act_bits);

/* Offline weight preparation (Sec. 4.2: fold D* into W, quantize to int4 with
 * symmetric steps, store packed integers with their scales).
 *   w        [N][K] fp32, the transposed weight W^T
 *   d        [K] fp32 positive channel scaling D, or NULL for D = I
 *   qw       out [N][K/2] packed int4 codes in [-7, 7]
 *   w_scale  out [K/w_group][N] fp16 steps (group-major)
 * Per (row j, group): w' = w * d[k]; Delta_W = fp16(amax|w'| / 7);
 * inv = 1 / fp32(Delta_W) (0 where infinite); code = rint(clamp(w' * inv, -7, 7)).
 * Requires amax / 7 <= 65504 in every group. */
sq_status sq_pack_weights(const float* w, const float* d, int32_t N, int32_t K, int32_t w_group,
                          uint8_t* qw, uint16_t* w_scale, hipStream_t stream);

/* The first kernel (Sec. 4.4): channel scaling, stream gain and quantization
 * of X [M][K] bf16 in one pass.
 *   act->act_bits == 8: qx = int8 [M][K]; act_scale = fp32 r [M]
 *   act->act_bits == 4: qx = packed int4 [M][K/2]; act_scale = fp16 sigma [M][K/64]
 * qx and act_scale must not overlap x. */
sq_status sq_quantize_act(const uint16_t* x, int32_t M, int32_t K, const sq_act_params* act,
                          void* qx, void* act_scale, hipStream_t stream);

/* The second kernel for 8-bit activations (Sec. 4.4, Eq. 10, with one int32
 * accumulator per K-block of w_group): C^b = Q_X Q_W over the block, then
 * Y_ij = r_i * sum_b fp32(C^b_ij) Delta_W[j][b] + b_j, cast to out_dtype.
 *   qx int8 [M][K], row_scale fp32 [M] (as written by sq_quantize_act),
 *   y  [M][N] of out_dtype.
 *   workspace: NULL (every output tile is computed whole) or a device buffer
 *   of ws_bytes (16-byte aligned; sq_workspace_bytes(SQ_VARIANT_GEMM, ...)
 *   enables the split-K tail) that must not overlap the other buffers. */
sq_status sq_gemm_w4a8(const int8_t* qx, const float* row_scale, int32_t M, const sq_weight* w,
                       void* y, int32_t out_dtype, void* workspace, size_t ws_bytes, hipStream_t stream);

/* The second kernel for 4-bit activations: one int32 accumulator per 64-wide
 * K-block, Y_ij = kappa_i * sum_b (fp32(C^b_ij) sigma_{i,b}) Delta_W[j][b(k)] + b_j
 * with kappa_i = 1 / gamma[tau][s(i)] (the inverse-gain compensation of Eq. 8,
 * taken from act->tok2stream, act->gamma and act->step).
 *   qx packed int4 [M][K/2], group_scale fp16 [M][K/64]; workspace as for
 *   sq_gemm_w4a8. */
sq_status sq_gemm_w4a4(const uint8_t* qx, const uint16_t* group_scale, int32_t M,
                       const sq_act_params* act, const sq_weight* w, void* y, int32_t out_dtype,
                       void* workspace, size_t ws_bytes, hipStream_t stream);

/* The fused linear with 8-bit activations: sq_quantize_act then sq_gemm_w4a8,
 * Q_X, r and the GEMM's partial sums living in `workspace`
 * (>= sq_workspace_bytes(SQ_VARIANT_FUSED, ...)).
 * Requires act->act_bits == 8 and w->K == K of x. */
sq_status sq_linear_w4a8(const uint16_t* x, int32_t M, const sq_act_params* act, const sq_weight* w,
                         void* y, int32_t out_dtype, void* workspace, size_t ws_bytes,
                         hipStream_t stream);

/* The fused linear with 4-bit activations (act->act_bits == 4).
 * With more than 128 tokens the codes go to gfx950's fp8 matrix cores
 * (v_mfma_f32_32x32x64_f8f6f4): the first kernel
 * writes each code as the fp8 e4m3 byte of code * 2^-9 (sign and magnitude;
 * |code| <= 7 is an exact subnormal), and the weight nibbles are read as
 * code + 8.  Products and block sums are exact in fp32, so the outputs equal
 * those of sq_quantize_act followed by sq_gemm_w4a4 bit for bit.
 * Workspace layout (each part 256-byte aligned, in this order): the codes
 * (fp8 bytes [M][K], else packed int4 [M][K/2]); sigma [M][K/64] (fp16, or
 * with fp8 codes its value as fp32); with fp8 codes kc fp32 [M][K/64] =
 * -8 S sigma 2^-18, S the code sum of the row's 64-group; then the GEMM's
 * partial sums.  With 8-bit activations:
 * Q_X int8 [M][K], r fp32 [M], partial sums. */
sq_status sq_linear_w4a4(const uint16_t* x, int32_t M, const sq_act_params* act, const sq_weight* w,
                         void* y, int32_t out_dtype, void* workspace, size_t ws_bytes,
                         hipStream_t stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the fused
 * W4A8 linear of sq_linear_w4a8 (same validation, kernels and results) with
 * no workspace argument.  Q_X, r and the GEMM's partial sums live in a device
 * array of SQ_NOALLOC_SCRATCH_BYTES inside this library, one per GPU, held
 * until the process ends; the call allocates and frees nothing.  Layers whose
 * sq_workspace_bytes(SQ_VARIANT_FUSED, M, K, N, 8) exceeds the array return
 * SQ_ERR_WORKSPACE and launch nothing.  Every call on a GPU shares that GPU's
 * array and leaves its contents behind (nothing in it needs to start at
 * zero): calls that overlap on one GPU (concurrent streams, or host threads
 * without ordering) race and must be serialized by the caller.  The first
 * call on each device looks the array's device address up (SQ_ERR_HIP if
 * that fails). */
#define SQ_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
sq_status sq_linear_w4a8_noalloc(const uint16_t* x, int32_t M, const sq_act_params* act, const sq_weight* w,
                                 void* y, int32_t out_dtype, hipStream_t stream);

/* The fused W4A8 linear as ONE kernel, for the paper's static activation
 * ranges (App. D: an offline threshold per layer and step) and few tokens:
 * the weight-streaming GEMM reads X itself and quantizes each 128-channel
 * stage in LDS with the first kernel's arithmetic (the quantization block of
 * this header, STATIC), so neither the first kernel's launch nor Q_X in HBM
 * remain (Sec. 4.4 on removing launches and intermediate traffic).  The
 * outputs equal those of sq_linear_w4a8 with the same arguments bit for bit.
 * Requires act->act_bits == 8, act->range_mode == SQ_RANGE_STATIC,
 * M <= 128 and w->w_group 128 or K (else SQ_ERR_UNSUPPORTED).
 *   workspace: NULL (K is never split across workgroups) or a device buffer
 *   of ws_bytes >= sq_workspace_bytes(SQ_VARIANT_GEMM, M, K, N, 8), 16-byte
 *   aligned, for the partial sums of a K split (contents need no
 *   initialization).
 * Every workgroup quantizes the activations it reads (M x its K range), so
 * the quantization work is repeated once per 32 output channels; with the
 * first kernel it is done once.  Which of the two is faster is measured. */
sq_status sq_linear_w4a8_static1(const uint16_t* x, int32_t M, const sq_act_params* act, const sq_weight* w,
                                 void* y, int32_t out_dtype, void* workspace, size_t ws_bytes, hipStream_t stream);

/* Producer-side fusion of the MLP's one direct chain, up projection -> GELU
 * -> down projection (the DiT block keeps GELU in bf16, App. D; Sec. 4.4 on
 * intermediate traffic): the fused W4A8 linear of the up projection (x, act,
 * w, workspace as for sq_linear_w4a8) whose GEMM epilogue does not store Y
 * but, per output, rounds Y to bf16, evaluates GELU with the sequence of
 * sq_gelu_bf16, rounds to bf16 and quantizes the result with the DOWN
 * projection's STATIC 8-bit quantizer (act_next: its stream ids, gains,
 * per-step thresholds, D^-1 and step; Eq. 1, 6 and 8).  Writes
 *   qx_next  int8 [M][N] (N = w->N = the down projection's K), 4-byte aligned
 *   r_next   fp32 [M], r_i = Delta / gamma_s(i) of the down layer,
 * exactly what sq_quantize_act(act_next) writes for the bf16 output of
 * sq_gelu_bf16 applied to sq_linear_w4a8's bf16 output; they feed
 * sq_gemm_w4a8 with the down projection's weights.  The down layer's
 * channel scaling act_next->dinv must be NULL or 16-byte aligned.
 * The epilogue runs in whichever GEMM the layer takes: the tiled one (more
 * than 128 tokens) or the weight-streaming one (at most 128 tokens), and in
 * the second kernel of a K split.
 * Requires act->act_bits == 8, w->w_group == 128 or K (one step per output
 * channel, the paper's weight format),
 * act_next->act_bits == 8 and act_next->range_mode == SQ_RANGE_STATIC (a
 * dynamic range needs the whole row before any code): else
 * SQ_ERR_UNSUPPORTED. */
sq_status sq_linear_w4a8_gelu_quant(const uint16_t* x, int32_t M, const sq_act_params* act, const sq_weight* w,
                                    const sq_act_params* act_next, int8_t* qx_next, float* r_next, void* workspace,
                                    size_t ws_bytes, hipStream_t stream);

/* The same producer-side fusion with 4-bit activations (the paper's W4A4
 * mode): the fused W4A4 linear of the up projection (x, act, w, workspace as
 * for sq_linear_w4a4) whose epilogue rounds Y to bf16, evaluates GELU as
 * sq_gelu_bf16 does, rounds to bf16 and quantizes with the DOWN projection's
 * STATIC 4-bit quantizer (act_next; Delta = fp16(clip[step] / 7), Eq. 1, 6
 * and 8).  It writes the down projection's first-kernel output in the form
 * that projection's GEMM takes at this token count:
 *   M <= 128  qx_next    packed int4 [M][N/2] (the layout of sq_quantize_act)
 *             scale_next fp16 sigma [M][N/64]; kc_next unused (may be NULL)
 *             -> sq_gemm_w4a4; equal, bit for bit, to what
 *             sq_quantize_act(act_next) writes for the bf16 output of
 *             sq_gelu_bf16 applied to sq_linear_w4a4's bf16 output;
 *   M > 128   qx_next    fp8 e4m3 code bytes [M][N] (code * 2^-9: sign and
 *                        magnitude, |code| <= 7, a zero code of a negative
 *                        value is -0)
 *             scale_next fp32 sigma [M][N/64] (the fp16 step, widened)
 *             kc_next    fp32 [M][N/64], -8 * S * sigma * 2^-18 with S the
 *                        sum of the row's 64 codes of the group
 *             -> sq_gemm_w4a4_fp8; the same codes and steps.
 * qx_next, scale_next and kc_next 4-byte aligned (scale_next 2-byte for
 * M <= 128).  The down layer's act_next->dinv must be NULL or 16-byte
 * aligned.  Requires act->act_bits == 4, act_next->act_bits == 4 and
 * act_next->range_mode == SQ_RANGE_STATIC (else SQ_ERR_UNSUPPORTED). */
sq_status sq_linear_w4a4_gelu_quant(const uint16_t* x, int32_t M, const sq_act_params* act, const sq_weight* w,
                                    const sq_act_params* act_next, void* qx_next, void* scale_next, float* kc_next,
                                    void* workspace, size_t ws_bytes, hipStream_t stream);

/* The second kernel on 4-bit activations in the fp8 form that
 * sq_linear_w4a4_gelu_quant writes for more than 128 tokens (Sec. 4.4 Eq.
 * 10 with 64-wide activation groups): fp8 code bytes qx [M][K] (16-byte
 * aligned), fp32 group steps sigma [M][K/64] and kc [M][K/64] (4-byte
 * aligned), on the fp8 matrix cores; the outputs equal sq_gemm_w4a4's on the
 * same codes and steps in the packed form.  act supplies the stream ids and
 * gains (kappa = 1 / gamma_s(i)) and act->act_bits must be 4.  M <= 128
 * returns SQ_ERR_UNSUPPORTED (sq_gemm_w4a4 takes the packed form there).
 * workspace as for sq_gemm_w4a4. */
sq_status sq_gemm_w4a4_fp8(const uint8_t* qx, const float* group_scale, const float* kc, int32_t M,
                           const sq_act_params* act, const sq_weight* w, void* y, int32_t out_dtype, void* workspace,
                           size_t ws_bytes, hipStream_t stream);

/* GELU of n bf16 values (x, y device buffers of n uint16 bit patterns,
 * 16-byte aligned, y may equal x; n may be 0): y = bf16(0.5 x (1 + erf(x /
 * sqrt 2))) with erf by Abramowitz and Stegun 7.1.28 as one fixed sequence of
 * fp32 operations (Horner's rule from a6, four squarings, 1 - 1/p), rounded
 * to nearest even; the op the quantized DiT keeps in bf16 (App. D). */
sq_status sq_gelu_bf16(const uint16_t* x, size_t n, uint16_t* y, hipStream_t stream);

/* The same layer without fusion, as the execution that Sec. 4.4 replaces:
 * channel scaling, gain, quantization, GEMM, dequantization, inverse-gain
 * compensation and bias each run as their own kernel, passing fp32 (or
 * int32) intermediates through `workspace`
 * (>= sq_workspace_bytes(SQ_VARIANT_UNFUSED, ...)).  act->act_bits 8 or 4.
 * Codes and accumulators equal the fused path's; outputs differ only in
 * fp32 rounding order. */
sq_status sq_linear_unfused(const uint16_t* x, int32_t M, const sq_act_params* act, const sq_weight* w,
                            void* y, int32_t out_dtype, void* workspace, size_t ws_bytes,
                            hipStream_t stream);

/* Activation calibration (Sec. 4.3, Eq. 9).  For a linear with fixed
 * quantized weights W^ = Q(D W), a candidate is one gain per stream
 * gamma_s and one threshold c shared by the streams; its objective is
 *
 *     L = sum_s omega_s / n_s * || gamma_s^-1 Q(gamma_s X~_s; c) W^ - X~_s W^ ||_F^2
 *
 * over the calibration tokens X (rows of stream s: X_s, n_s of them), with
 * X~ = X D^-1.  A stream with no token adds nothing.  The search over
 * candidates is the caller's: evaluate a batch, keep the smallest.
 *
 * sq_calib_reference writes the target X~ W^ once per linear:
 * y_ref[i][j] = sum_k x~_ik * code_jk * Delta_W, in fp64 (each product
 * exact, x~ = fp32(x) * dinv rounded to fp32 as in the quantizer), fp64
 * [M, N] row-major, 16-byte aligned.  dinv [K] as in sq_act_params (NULL:
 * D = I).  w->bias is not used. */
sq_status sq_calib_reference(const uint16_t* x, int32_t M, const float* dinv, const sq_weight* w, double* y_ref,
                             hipStream_t stream);

/* Bytes of device workspace for sq_calib_objective with this shape, bits
 * and stream count (1 <= num_streams <= 4096); 0 for invalid arguments.
 * Host-only. */
size_t sq_calib_workspace_bytes(int32_t M, int32_t K, int32_t N, int32_t act_bits, int32_t num_streams);

/* Evaluates L for num_candidates (1 .. 65536) candidates, in order:
 *   cand_gamma  fp32 [num_candidates][num_streams]  gains, finite and > 0
 *   cand_clip   fp32 [num_candidates]               thresholds c > 0
 *   omega       fp64 [num_streams]                  stream weights (uniform: 1/S)
 *   objective   fp64 [num_candidates]               out
 * x, M, tok2stream, dinv and act_bits as for sq_linear_w4a8 / sq_linear_w4a4;
 * y_ref from sq_calib_reference with the same x, dinv and w.  Each candidate
 * runs the fused linear in STATIC range mode with the one-step tables
 * (gamma, c), without the bias (it cancels), into fp32 Y_c, then
 * L = sum_i omega_s(i) / n_s(i) * sum_j (Y_c,ij - y_ref,ij)^2, accumulated in
 * fp64 in a fixed order (the result is reproducible).  Y_c differs from the
 * exact modulated product by the fused linear's fp32 rounding.  Alignment:
 * x, y_ref and workspace 16 bytes, omega and objective 8, the rest 4.
 * Candidates are enqueued one after another on `stream`; a launch failure
 * returns SQ_ERR_HIP after the earlier candidates were enqueued. */
sq_status sq_calib_objective(const uint16_t* x, int32_t M, const int32_t* tok2stream, int32_t num_streams,
                             const float* dinv, int32_t act_bits, const sq_weight* w, const double* y_ref,
                             int32_t num_candidates, const float* cand_gamma, const float* cand_clip,
                             const double* omega, double* objective, void* workspace, size_t workspace_bytes,
                             hipStream_t stream);

/* Shared channel scaling, Sec. 4.2 Eq. 7.  The paper chooses D* by
 *
 *     L(D) = sum_r weight_r / n_r * || Q(X_r D^-1) Q(D W) - X_r W ||_F^2
 *
 * over regions r (per step and stream; weight_r = pi_tau omega^D_{tau,s})
 * but names no family for D and no optimizer.  This library evaluates the
 * one-parameter family d_k = amax_i |x_ik|^alpha / amax_j |w_jk|^(1 - alpha)
 * (fp64, clamped to [2^-6, 2^6], then fp32; 1 where either amax is 0) for a
 * list of exponents; the caller keeps the best and folds it with
 * sq_pack_weights.
 *
 * sq_calib_fp_reference writes the full-precision target Y = X W^T in fp64:
 * x bf16 [M, K], w fp32 [N, K] (16-byte aligned), y_ref fp64 [M, N]. */
sq_status sq_calib_fp_reference(const uint16_t* x, int32_t M, const float* w, int32_t N, int32_t K, double* y_ref,
                                hipStream_t stream);

/* d fp32 [K] and dinv = fp32(1 / d) [K] of the family above for one alpha
 * (finite), from the per-channel maxima of |x| over the M rows of x (bf16
 * [M, K]) and of |w| over the N rows of w (fp32 [N, K], 1 <= N <= 2^20).
 * d and dinv must be distinct; they also serve as scratch.  x and w 16-byte
 * aligned. */
sq_status sq_smooth_scales(const uint16_t* x, int32_t M, const float* w, int32_t N, int32_t K, float alpha, float* d,
                           float* dinv, hipStream_t stream);

/* Workspace bytes for sq_calib_scaling_objective (1 <= num_regions <= 4096);
 * 0 for invalid arguments.  Host-only. */
size_t sq_calib_scaling_workspace_bytes(int32_t M, int32_t K, int32_t N, int32_t w_group, int32_t act_bits,
                                        int32_t num_regions);

/* L(D) of Eq. 7 for each exponent alphas[i] (a HOST array of num_alphas
 * finite values, 1 .. 65536) into objective[i] (device fp64):
 *   region         int32 [M], the region of every row; each must lie in
 *                  [0, num_regions) (device data, not checked, as tok2stream)
 *   region_weight  fp64 [num_regions] (device)
 *   w              fp32 [N, K] the unquantized weight; y_ref its target from
 *                  sq_calib_fp_reference
 * Per exponent: d and dinv as sq_smooth_scales, Q(D W) packed with w_group,
 * then the fused linear with DYNAMIC ranges (per token for act_bits 8, per 64
 * channels for 4), unit gains and no bias into fp32, and the weighted squared
 * error in fp64 in a fixed order.  Alignment: x, w, y_ref and workspace 16
 * bytes, region_weight and objective 8, region 4. */
sq_status sq_calib_scaling_objective(const uint16_t* x, int32_t M, const int32_t* region, int32_t num_regions,
                                     const double* region_weight, const float* w, int32_t N, int32_t K,
                                     int32_t w_group, int32_t act_bits, const double* y_ref, int32_t num_alphas,
                                     const float* alphas, double* objective, void* workspace, size_t workspace_bytes,
                                     hipStream_t stream);

/* Constrained search for (gamma*, c*) of Eq. 9 under the constraints of
 * Sec. 4.3 and App. C.1: gamma_min <= gamma_s <= gamma_max for every stream,
 * clip_min <= c <= clip_max and sum_s n_s log gamma_s = 0.  The paper names
 * no optimizer; this one is a compass search in log coordinates
 * (log gamma_1 .. log gamma_S, log c) started at gamma = 1 (which meets every
 * constraint) and c = clip_init clamped to its bounds, with step log_step.
 * Each round tries, for every coordinate in turn (the S gains, then c), a
 * step of +h and of -h: 2 (S + 1) candidates.  A gain step is mapped back
 * onto the constraint set by the nearest point in the token-weighted norm
 * sum_s n_s (u_s - v_s)^2 (u_s = clamp(v_s - lambda), lambda found by 64
 * bisection halvings in fp64; a stream without tokens is only clamped); a
 * threshold step is clamped.  Gains and thresholds are evaluated as fp32
 * values exp(.) clamped to the bounds.  The first candidate with the smallest
 * objective replaces the incumbent when strictly better; otherwise h halves.
 * Everything, including the search state, stays on the device: the call
 * enqueues `rounds` rounds and returns without synchronizing. */
typedef struct sq_calib_search_params {
  float gamma_min, gamma_max; /* 0 < gamma_min <= 1 <= gamma_max */
  float clip_min, clip_max;   /* 0 < clip_min <= clip_max */
  float clip_init;            /* start threshold (finite) */
  float log_step;             /* initial step h in log space, 0 < h <= 64 (the projection's 64
                                 bisection halvings then resolve lambda to fp64 precision) */
  int32_t rounds;             /* 0 .. 1024 (0: evaluate the start only) */
} sq_calib_search_params;

/* Workspace bytes for sq_calib_search (1 <= num_streams <= 64); 0 for
 * invalid arguments.  Host-only. */
size_t sq_calib_search_workspace_bytes(int32_t M, int32_t K, int32_t N, int32_t act_bits, int32_t num_streams);

/* Arguments as for sq_calib_objective; params is a host struct.  Outputs
 * (device): gamma_out fp32 [num_streams], clip_out fp32 [1] and
 * objective_out fp64 [1], the best point found and its objective, which is
 * bit-identical to what sq_calib_objective returns for that point.  The
 * outputs also hold the incumbent during the search.  Non-finite or
 * inconsistent bounds return SQ_ERR_UNSUPPORTED. */
sq_status sq_calib_search(const uint16_t* x, int32_t M, const int32_t* tok2stream, int32_t num_streams,
                          const float* dinv, int32_t act_bits, const sq_weight* w, const double* y_ref,
                          const double* omega, const sq_calib_search_params* params, float* gamma_out,
                          float* clip_out, double* objective_out, void* workspace, size_t workspace_bytes,
                          hipStream_t stream);

/* Measurement hook: the int8 matrix-core rate the GPU sustains, as a
 * ceiling beside the published peak.  Launches sq_probe_mfma_i8_sink_bytes()
 * / 1024 workgroups (two per CU) whose waves each issue back-to-back int8
 * MFMAs on register operands, with no memory traffic, 2^20 int8 operations
 * per wave and iteration:
 *   shape 32: iters * 16 v_mfma_i32_32x32x32_i8 (four 32 x 32 tiles); with
 *             fold != 0 each tile's accumulator is also converted and fma'd
 *             into fp32 once per four MFMAs (one 128-channel block);
 *   shape 16: iters * 32 v_mfma_i32_16x16x64_i8 (sixteen 16 x 16 tiles of
 *             two MFMAs); with fold != 0 each block starts from the integer
 *             bits of 1.5 * 2^23 and is folded by a subtraction and an fma
 *             per output, as the 16 x 16 tiled GEMM does.
 * Operands all zero (random_operands == 0) or pseudo-random.  The caller
 * times the call (e.g. with HIP events); sink is int32 scratch of at least
 * sq_probe_mfma_i8_sink_bytes() bytes that keeps the work live.
 * iters in [1, 2^24]; another shape returns SQ_ERR_UNSUPPORTED. */
size_t sq_probe_mfma_i8_sink_bytes(void);
sq_status sq_probe_mfma_i8(int32_t shape, int32_t iters, int32_t random_operands, int32_t fold, int32_t* sink,
                           size_t sink_bytes, hipStream_t stream);

/* Measurement hook for the 4-bit path's matrix-core instruction,
 * v_mfma_scale_f32_32x32x64_f8f6f4, with fp8 e4m3 (format 8) or fp6 e2m3
 * (format 6) operands: the same grid as sq_probe_mfma_i8, each wave issuing
 * iters * 8 MFMAs on register operands (2^20 operations per iteration: the
 * eight MFMAs of one 128-channel stage of the fp8 W4A4 GEMM).  With fold != 0
 * every block's fp32 sum is also folded by two fmas per output, as that GEMM
 * does.  Operands all zero or pseudo-random (fp8 bytes without NaN codes).
 * sink: int32 scratch of sq_probe_mfma_i8_sink_bytes() bytes; iters in
 * [1, 2^24]; another format returns SQ_ERR_UNSUPPORTED. */
sq_status sq_probe_mfma_f8f6(int32_t format, int32_t iters, int32_t random_operands, int32_t fold, int32_t* sink,
                             size_t sink_bytes, hipStream_t stream);

/* Test hook: writes every int32 block accumulator of Q_X Q_W instead of an
 * epilogue: acc_out[b][i][j] = sum over K-block b of q_ik * w_jk, with blocks
 * of w_group (8-bit) or 64 (4-bit).  It runs the library's non-pipelined GEMM
 * kernel (the one that serves 8-bit activations with 128 < w_group < K and
 * the unfused path's int32 C), NOT the kernels the fused linear normally
 * dispatches to (the pipelined int8 and fp8 kernels and the weight-streaming
 * kernel); those have no dump epilogue, and their block sums are checked
 * through outputs computed in exact arithmetic instead (integer activations,
 * power-of-two steps).  qx as for sq_gemm_w4a8 / sq_gemm_w4a4.
 * acc_out is int32 [K/block][M][N]. */
sq_status sq_debug_block_acc_i32(const void* qx, int32_t M, int32_t act_bits, const sq_weight* w,
                                 int32_t* acc_out, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* SQ_H_ */
