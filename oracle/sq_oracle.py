"""CPU oracle for the fused low-bit linear of a world-action DiT (SteerQuant /
Rudder, arXiv 2609.39056).  TEST INFRASTRUCTURE ONLY: the tests, the smoke
check and the benchmark's CPU-baseline leg may call it; the product path never
does.

Plain, slow and step-by-step.  Every floating-point step is an IEEE binary32
operation with round-to-nearest-even, evaluated in exactly the order written
(numpy float32 arrays: one rounding per operation, no fused multiply-add).  The
integer GEMM is exact.  Nothing here is shared with the HIP implementation.

What is computed, following the paper:

* Symmetric k-bit quantizer, Sec. 3.1 Eq. (1): Q = clip(round(X / Delta),
  -q_max, q_max) with Delta = c / q_max and q_max = 2^(k-1) - 1.
* Channel scaling, Sec. 4.2 Eq. (6): the input is X D^-1 and the weight is
  Q(D W); one D per layer, shared by all streams and steps.
* Stream-specific modulation, Sec. 4.3 Eq. (8): gamma^-1 Q(gamma X D^-1; c) W^.
* Rudder's two kernels, Sec. 4.4: the first applies D^-1 and the stream gain
  while quantizing and emits integer activations plus row scales
  r_i = Delta_X / gamma_s(i); the second accumulates Q_X Q_W in INT32 and
  applies Eq. (10): Y = cast[(FP32(C_ij) r_i) Delta_W,j + b_j].
* Effective ranges, App. C.1: stream s sees threshold c / gamma_s.

Readings where the paper leaves a choice:

* Two range modes.  STATIC: c is the per-step table value c_tau (the paper's
  static activation scale, App. D).  DYNAMIC: c is the absolute maximum of
  X D^-1 over the row (A8) or over a 64-wide group of the row (A4), taken
  before the gain, so the gain still moves the effective threshold to c/gamma.
* Quantizing divides by multiplying with a reciprocal:
  Delta = c / q_max, inv = 1 / Delta, t = (x~ * g) * inv.  If 1 / Delta is
  infinite (Delta = 0 or tiny), inv = 0 and the codes are 0.
* Rounding is round-half-to-even; clamping happens in float before rounding.
* A4 steps are rounded to fp16 before use (Delta <- fp16(Delta)), so the
  stored fp16 group scale is exactly the quantization step, and the gain
  compensation gamma^-1 (kappa) is applied per row in the epilogue.
* Weights may carry one fp16 scale per output channel (group = K, as in the
  paper) or per 128-wide group of K.  The epilogue then sums, over K-blocks in
  ascending order, (FP32(C_block) * s) * Delta_W; with a single block this is
  Eq. (10) exactly.
* Calibration, Sec. 4.3 Eq. (9): the paper gives the objective and its
  constraints but no optimizer; the search here is a compass search in log
  coordinates with every trial point projected onto the constraint set (the
  token-weighted nearest point) and the step halved after a round without
  progress.
* Shared scaling, Sec. 4.2 Eq. (7): the paper gives the objective but no
  family for D and no optimizer; the family here is d_k = amax|X_k|^alpha /
  amax|W_k|^(1-alpha) (clamped to [2^-6, 2^6]) over a list of exponents, with
  the per-token / per-group absmax activation quantizer and unit gains.
* MLP chain (producer-side fusion of the up projection into the down
  projection's quantizer): the up output is cast to bf16 as the layer's output
  would be, GELU is evaluated on that bf16 value and rounded to bf16 (GELU
  stays in BF16, App. D), and the result is the down projection's input,
  quantized with its STATIC thresholds.  GELU(x) = x Phi(x) =
  0.5 x (1 + erf(x / sqrt 2)); the paper does not say how erf is evaluated,
  so erf here is the rational approximation 7.1.28 of Abramowitz & Stegun
  (erf z ~ 1 - (1 + a1 z + ... + a6 z^6)^-16, |error| <= 3e-7), written as a
  fixed sequence of fp32 operations.
* int4 packing (both weights and A4 activations): for every 8 consecutive
  codes k = 8g..8g+7 the four bytes 4g..4g+3 hold code 8g+b in the low nibble
  and code 8g+b+4 in the high nibble of byte 4g+b.
"""
from __future__ import annotations

import numpy as np

RANGE_DYNAMIC = 0
RANGE_STATIC = 1
A4_GROUP = 64
Q_MAX = {8: 127, 4: 7}
W_QMAX = 7

F32 = np.float32


# --------------------------------------------------------------------------
# Number formats
# --------------------------------------------------------------------------
def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to fp32."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(F32)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 with round-to-nearest-even (finite inputs)."""
    u = np.ascontiguousarray(x, dtype=F32).view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    r = (u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)
    return (r & np.uint64(0xFFFF)).astype(np.uint16)


def f16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return np.asarray(bits, dtype=np.uint16).view(np.float16).astype(F32)


def f32_to_f16_bits(x: np.ndarray) -> np.ndarray:
    """fp32 -> fp16 with round-to-nearest-even (numpy's IEEE conversion)."""
    with np.errstate(over="ignore"):
        return np.asarray(x, dtype=F32).astype(np.float16).view(np.uint16)


def pack_int4(codes: np.ndarray) -> np.ndarray:
    """Pack int codes in [-8, 7], shape [R, K] (K % 8 == 0), to bytes [R, K/2].

    Byte 4g+b holds code 8g+b (low nibble) and code 8g+b+4 (high nibble)."""
    c = np.asarray(codes).astype(np.int64)
    R, K = c.shape
    assert K % 8 == 0
    nib = (c & 0xF).astype(np.uint8).reshape(R, K // 8, 2, 4)
    lo, hi = nib[:, :, 0, :], nib[:, :, 1, :]
    return (lo | (hi << np.uint8(4))).reshape(R, K // 2)


def unpack_int4(packed: np.ndarray) -> np.ndarray:
    """Inverse of pack_int4: bytes [R, K/2] -> int8 codes [R, K] (two's
    complement nibbles, -8..7)."""
    p = np.asarray(packed, dtype=np.uint8)
    R, H = p.shape
    g = p.reshape(R, H // 4, 4)
    lo = (g & np.uint8(0xF)).astype(np.int16)
    hi = (g >> np.uint8(4)).astype(np.int16)
    both = np.stack([lo, hi], axis=2)                    # [R, H/4, 2, 4]
    signed = np.where(both >= 8, both - 16, both)
    return signed.reshape(R, H * 2).astype(np.int8)


# --------------------------------------------------------------------------
# First kernel: channel scaling, stream gain, quantization (Sec. 4.4, first
# kernel; Eq. (1) applied to gamma X D^-1 as in Eq. (8))
# --------------------------------------------------------------------------
def _reciprocal_or_zero(delta: np.ndarray) -> np.ndarray:
    with np.errstate(divide="ignore", over="ignore"):
        inv = F32(1.0) / delta
    return np.where(np.isinf(inv), F32(0.0), inv).astype(F32)


def quantize_act(x_bits, tok2stream, gamma, step, dinv=None, clip=None,
                 range_mode=RANGE_DYNAMIC, act_bits=8):
    """Quantize bf16 activations [M, K] for one layer at denoising step `step`.

    Returns a dict with
      codes  int8 [M, K]          the integer activations Q_X
      qx     A8: int8 [M, K]; A4: uint8 [M, K/2] packed (the stored form)
      scale  A8: fp32 r [M]  (r_i = Delta_i / gamma_s(i), Sec. 4.4)
             A4: fp16 bit patterns sigma [M, K/64] (the fp16 step per group)
      kappa  fp32 [M], 1 / gamma_s(i) (the output compensation of Eq. (8))
      delta  fp32 [M, groups] the quantization step per row / group
      xt     fp32 [M, K] the channel-scaled activation X D^-1
      g      fp32 [M] the row's gain
    """
    x_bits = np.asarray(x_bits, dtype=np.uint16)
    M, K = x_bits.shape
    qa = Q_MAX[act_bits]
    gamma = np.asarray(gamma, dtype=F32)
    S = gamma.shape[1]
    t2s = np.asarray(tok2stream, dtype=np.int64)
    assert t2s.shape == (M,)
    assert np.all((t2s >= 0) & (t2s < S)), "stream id out of range"
    assert 0 <= step < gamma.shape[0]

    # Row gain gamma_{tau, s(i)} (Sec. 4.3; the token-wise diagonal of Fig. 2).
    g = gamma[step, t2s].astype(F32)

    # Channel scaling X D^-1 (Eq. 6), one fp32 multiply per element.
    x = bf16_bits_to_f32(x_bits)
    xt = x if dinv is None else (x * np.asarray(dinv, dtype=F32)[None, :]).astype(F32)

    group = K if act_bits == 8 else A4_GROUP
    assert K % group == 0
    ng = K // group
    xg = xt.reshape(M, ng, group)

    # Reference range c: the per-step table value, or the group's amax of
    # X D^-1 before the gain.
    if range_mode == RANGE_STATIC:
        assert clip is not None
        c = np.full((M, ng), np.asarray(clip, dtype=F32)[step], dtype=F32)
    else:
        c = np.max(np.abs(xg), axis=2).astype(F32)

    # Step Delta = c / q_max (Eq. 1).  A4 steps are fp16 values.
    delta = (c / F32(qa)).astype(F32)
    if act_bits == 4:
        delta = f16_bits_to_f32(f32_to_f16_bits(delta))
    inv = _reciprocal_or_zero(delta)

    # t = (x~ * gamma) * (1 / Delta); clamp to [-q_max, q_max]; round to even.
    t = ((xg * g[:, None, None]).astype(F32) * inv[:, :, None]).astype(F32)
    t = np.minimum(np.maximum(t, F32(-qa)), F32(qa))
    codes = np.rint(t).astype(np.int8).reshape(M, K)

    kappa = (F32(1.0) / g).astype(F32)
    if act_bits == 8:
        r = (delta[:, 0] / g).astype(F32)          # r_i = Delta_X / gamma_s(i)
        return dict(codes=codes, qx=codes.copy(), scale=r, kappa=kappa,
                    delta=delta, xt=xt, g=g)
    sigma = f32_to_f16_bits(delta)
    return dict(codes=codes, qx=pack_int4(codes), scale=sigma, kappa=kappa,
                delta=delta, xt=xt, g=g)


# --------------------------------------------------------------------------
# Offline weight preparation: fold D, quantize per group to int4, pack
# (Sec. 4.2: the channel scaling is folded into the weights, which are then
# kept as packed integers)
# --------------------------------------------------------------------------
def pack_weights(w, d=None, w_group=128):
    """w: fp32 [N, K] (W^T), d: fp32 [K] or None.

    Returns codes int8 [N, K] in [-7, 7], qw uint8 [N, K/2] (packed), and
    w_scale fp16 bit patterns [N, K / w_group]."""
    w = np.asarray(w, dtype=F32)
    N, K = w.shape
    assert K % w_group == 0
    wf = w if d is None else (w * np.asarray(d, dtype=F32)[None, :]).astype(F32)
    nb = K // w_group
    wg = wf.reshape(N, nb, w_group)
    amax = np.max(np.abs(wg), axis=2).astype(F32)
    scale_bits = f32_to_f16_bits((amax / F32(W_QMAX)).astype(F32))
    inv = _reciprocal_or_zero(f16_bits_to_f32(scale_bits))
    t = (wg * inv[:, :, None]).astype(F32)
    t = np.minimum(np.maximum(t, F32(-W_QMAX)), F32(W_QMAX))
    codes = np.rint(t).astype(np.int8).reshape(N, K)
    return dict(codes=codes, qw=pack_int4(codes), w_scale=scale_bits)


# --------------------------------------------------------------------------
# Second kernel: INT32 accumulation and the dequantization epilogue
# (Sec. 4.4, Eq. (10), generalized to K-blocks)
# --------------------------------------------------------------------------
def block_size(act_bits: int, K: int, w_group: int) -> int:
    """K-block over which one int32 accumulator runs: the smaller of the
    activation group (K for A8, 64 for A4) and the weight group."""
    return min(K if act_bits == 8 else A4_GROUP, w_group)


def block_acc(codes_x, codes_w, G):
    """C^beta_ij = sum_{k in block beta} q_ik w_jk, exactly.

    codes_x int [M, K], codes_w int [N, K] -> int64 [K/G, M, N].  The float64
    matmul is exact: every partial sum is an integer below 2^53."""
    qx = np.asarray(codes_x, dtype=np.float64)
    qw = np.asarray(codes_w, dtype=np.float64)
    M, K = qx.shape
    assert K % G == 0
    out = np.empty((K // G, M, qw.shape[0]), dtype=np.int64)
    for b in range(K // G):
        sl = slice(b * G, (b + 1) * G)
        blk = qx[:, sl] @ qw[:, sl].T
        out[b] = blk.astype(np.int64)
    assert np.abs(out).max(initial=0) < 2**31, "int32 accumulator overflow"
    return out


def epilogue(C, act_bits, scale, kappa, w_scale_bits, w_group, bias_bits=None):
    """Dequantize block accumulators C [nb, M, N] (int64) into fp32 y.

    A8: y = sum_beta (f32(C^beta) * r_i) * Delta_W[j, beta]        (+ b_j)
    A4: y = (sum_beta (f32(C^beta) * sigma_i,beta) * Delta_W[j, b(beta)]) * kappa_i  (+ b_j)

    Also returns y64 (the same sum in fp64) and A (sum of the magnitudes of
    the terms, the scale of the rounding error)."""
    nb, M, N = C.shape
    K = None
    ws = f16_bits_to_f32(w_scale_bits)                       # [N, K/w_group]
    n_wg = ws.shape[1]
    K = n_wg * w_group
    G = K // nb
    y = np.zeros((M, N), dtype=F32)
    y64 = np.zeros((M, N), dtype=np.float64)
    A = np.zeros((M, N), dtype=np.float64)
    if act_bits == 8:
        s_all = np.asarray(scale, dtype=F32)[:, None]         # r_i, [M, 1]
    else:
        sig = f16_bits_to_f32(scale)                          # [M, K/64]
    for b in range(nb):
        wb = (b * G) // w_group
        dw = ws[:, wb][None, :]                               # [1, N]
        s = s_all if act_bits == 8 else sig[:, b][:, None]
        term = ((C[b].astype(F32) * s).astype(F32) * dw).astype(F32)
        y = (y + term).astype(F32)
        t64 = C[b].astype(np.float64) * s.astype(np.float64) * dw.astype(np.float64)
        y64 += t64
        A += np.abs(t64)
    if act_bits == 4:
        k = np.asarray(kappa, dtype=F32)[:, None]
        y = (y * k).astype(F32)
        y64 *= k.astype(np.float64)
        A *= k.astype(np.float64)
    if bias_bits is not None:
        b32 = bf16_bits_to_f32(bias_bits)[None, :]
        y = (y + b32).astype(F32)
        y64 += b32.astype(np.float64)
        A += np.abs(b32.astype(np.float64))
    return y, y64, A


def cast_output(y, out_dtype):
    """'f32' -> fp32 values; 'bf16' / 'f16' -> bit patterns (uint16)."""
    if out_dtype == "f32":
        return np.asarray(y, dtype=F32)
    if out_dtype == "bf16":
        return f32_to_bf16_bits(y)
    if out_dtype == "f16":
        return f32_to_f16_bits(y)
    raise ValueError(out_dtype)


def linear(x_bits, tok2stream, gamma, step, qw_codes, w_scale_bits, w_group,
           dinv=None, clip=None, bias_bits=None, range_mode=RANGE_DYNAMIC, act_bits=8):
    """The whole fused linear: quantize (first kernel), block accumulate and
    epilogue (second kernel).  Returns the quantize dict plus C, y, y64, A."""
    qa = quantize_act(x_bits, tok2stream, gamma, step, dinv=dinv, clip=clip,
                      range_mode=range_mode, act_bits=act_bits)
    K = qa["codes"].shape[1]
    G = block_size(act_bits, K, w_group)
    C = block_acc(qa["codes"], qw_codes, G)
    y, y64, A = epilogue(C, act_bits, qa["scale"], qa["kappa"], w_scale_bits, w_group, bias_bits)
    qa.update(C=C, y=y, y64=y64, A=A, G=G)
    return qa


def full_precision_linear(x_bits, w, bias_bits=None):
    """Y = X W (+ b) in fp64 with unquantized operands (the target of Eq. 2)."""
    y = bf16_bits_to_f32(x_bits).astype(np.float64) @ np.asarray(w, np.float64).T
    if bias_bits is not None:
        y = y + bf16_bits_to_f32(bias_bits).astype(np.float64)[None, :]
    return y


# --------------------------------------------------------------------------
# GELU between the up and down projections of the MLP, in bf16 (App. D), and
# the chain into the down projection's STATIC quantizer (Sec. 4.4, the
# producer-side fusion of the intermediate activation)
# --------------------------------------------------------------------------
# Abramowitz & Stegun 7.1.28: erf z ~ 1 - (1 + a1 z + a2 z^2 + ... + a6 z^6)^-16
AS_ERF_COEFFS = (0.0705230784, 0.0422820123, 0.0092705272, 0.0001520143, 0.0002765672, 0.0000430638)
INV_SQRT2 = F32(0.70710677)  # fp32(1 / sqrt 2)


def erf_as(z):
    """erf of z >= 0 (fp32 array) by 7.1.28, one IEEE fp32 operation at a
    time: the polynomial by Horner's rule from a6 down, the 16th power by four
    squarings, then 1 - 1 / p^16 (0 where p^16 overflows to infinity)."""
    z = np.asarray(z, dtype=F32)
    a = [F32(c) for c in AS_ERF_COEFFS]
    p = np.full(z.shape, a[5], dtype=F32)
    with np.errstate(over="ignore", divide="ignore"):  # large z: p overflows to +inf and 1 / p to 0
        for c in (a[4], a[3], a[2], a[1], a[0], F32(1.0)):
            p = ((p * z).astype(F32) + c).astype(F32)
        for _ in range(4):
            p = (p * p).astype(F32)
        inv = (F32(1.0) / p).astype(F32)
    return (F32(1.0) - inv).astype(F32)


def gelu_f32(x):
    """GELU of fp32 x: 0.5 x (1 + erf(x / sqrt 2)) with the erf above, as
    z = |x| * fp32(1/sqrt 2), e = erf(z), s = 1 + e (x >= 0) or 1 - e
    (x < 0), then x * (s * 0.5) (the halving is exact, and taken first so
    that x * s cannot overflow)."""
    x = np.asarray(x, dtype=F32)
    with np.errstate(invalid="ignore"):  # NaN inputs, and -inf * 0, give NaN
        e = erf_as((np.abs(x) * INV_SQRT2).astype(F32))
        s = np.where(x >= 0, (F32(1.0) + e).astype(F32), (F32(1.0) - e).astype(F32)).astype(F32)
        return (x * (s * F32(0.5)).astype(F32)).astype(F32)


def gelu_bf16(h_bits):
    """GELU on bf16 values (bit patterns), rounded to bf16 (RNE)."""
    return f32_to_bf16_bits(gelu_f32(bf16_bits_to_f32(h_bits)))


def mlp_chain_codes(y_up, tok2stream, gamma_down, step, dinv_down, clip_down, act_bits=8):
    """The down projection's codes and scales (8-bit: row scales; 4-bit:
    fp16 group steps) from the up projection's fp32 output y_up [M, N_up]:
    cast to bf16 (the layer's output format), GELU in bf16, then the STATIC
    quantizer of the down layer (its gains, thresholds and D^-1; Eq. 1, 6,
    8).  Returns (h, g, qa): the up output in bf16, the GELU output in bf16
    and quantize_act's result."""
    h = f32_to_bf16_bits(np.asarray(y_up, dtype=F32))
    g = gelu_bf16(h)
    qa = quantize_act(g, tok2stream, gamma_down, step, dinv=dinv_down, clip=clip_down,
                      range_mode=RANGE_STATIC, act_bits=act_bits)
    return h, g, qa


# --------------------------------------------------------------------------
# Activation calibration objective, Sec. 4.3 Eq. (9)
# --------------------------------------------------------------------------
def calib_reference(x_bits, qw_codes, w_scale_bits, w_group, dinv=None):
    """The target of Eq. (9): X~ W^ with the activations unquantized,
    X~ = X D^-1 (the fp32 product of the quantizer's first step), and the
    fixed quantized weights W^ = code * Delta_W.  float64 [M, N]; every
    product is exact in float64 and the sums carry float64 rounding only."""
    x = bf16_bits_to_f32(np.asarray(x_bits, dtype=np.uint16))
    if dinv is not None:
        x = (x * np.asarray(dinv, dtype=F32)[None, :]).astype(F32)
    codes = np.asarray(qw_codes, dtype=np.int64)
    N, K = codes.shape
    steps = f16_bits_to_f32(w_scale_bits).astype(np.float64)   # [N, K / w_group]
    wq = codes.astype(np.float64) * np.repeat(steps, w_group, axis=1)[:, :K]
    return x.astype(np.float64) @ wq.T


def calib_objective(x_bits, tok2stream, num_streams, qw_codes, w_scale_bits, w_group, gammas, clips,
                    omega, dinv=None, act_bits=8, ref=None):
    """Eq. (9) for each candidate (gamma_s for every stream, shared threshold c):

        L = sum_s omega_s / n_s * || gamma_s^-1 Q(gamma_s X~_s; c) W^ - X~_s W^ ||_F^2

    The modulated output is the STATIC linear with the one-step gain table
    [gamma] and clip [c], taken at its float64 value (y64: exact block sums
    and the stored fp32 scales, no bias); n_s counts the tokens of stream s,
    and a stream with none adds 0.  omega holds the map weights (uniform:
    1 / S).  Returns float64 [n_candidates]."""
    if ref is None:
        ref = calib_reference(x_bits, qw_codes, w_scale_bits, w_group, dinv)
    t2s = np.asarray(tok2stream)
    out = []
    for g, c in zip(np.asarray(gammas, dtype=F32), np.asarray(clips, dtype=F32)):
        res = linear(x_bits, t2s, g[None, :], 0, qw_codes, w_scale_bits, w_group, dinv=dinv,
                     clip=np.array([c], dtype=F32), bias_bits=None, range_mode=RANGE_STATIC, act_bits=act_bits)
        out.append(weighted_stream_error(res["y64"], ref, t2s, num_streams, omega))
    return np.array(out, dtype=np.float64)


def weighted_stream_error(y, ref, ids, num_ids, omega):
    """sum_s omega_s / n_s * sum_{i : ids_i = s} || y_i - ref_i ||^2 (float64):
    each stream's (or region's) mean squared row error, weighted; a stream
    with no rows adds 0 (Eq. (7) and (9))."""
    d2 = ((np.asarray(y, np.float64) - ref) ** 2).sum(axis=1)
    ids = np.asarray(ids)
    L = 0.0
    for s in range(num_ids):
        rows = ids == s
        n = int(rows.sum())
        if n:
            L += float(omega[s]) / n * float(d2[rows].sum())
    return L


# ---------------------------------------------------------------- constrained search, Eq. (9)
# Sec. 4.3 (the constraints under Eq. (9)) and App. C.1 fix the constraints of
# the joint (gamma, c) calibration (bounds on c and on every gamma_s, and
# sum_s n_s log gamma_s = 0, which makes c the token-weighted geometric mean
# of the effective thresholds c / gamma_s) but name no search procedure.  The reading here: a compass (pattern) search in the log
# coordinates (log gamma_1 .. log gamma_S, log c), each trial point projected
# back onto the constraint set, with the step halved after a round that finds
# no better point.

def project_log_gains(v, counts, lo, hi, iters=64):
    """The point u nearest to v in the token-weighted norm sum_s n_s (u_s - v_s)^2
    with lo <= u_s <= hi and sum_s n_s u_s = 0 (lo <= 0 <= hi).  By the KKT
    conditions u_s = clamp(v_s - lam, lo, hi) for the streams with tokens; the
    sum is non-increasing in lam, and lam is found by bisection in float64 (a
    fixed number of halvings).  A stream without tokens is only clamped."""
    v = np.asarray(v, dtype=np.float64)
    n = np.asarray(counts, dtype=np.float64)
    live = n > 0
    if not live.any():
        return np.clip(v, lo, hi)

    def f(lam):   # summed stream by stream, in order
        t = 0.0
        for s in np.flatnonzero(live):
            t += float(n[s]) * min(max(float(v[s]) - lam, lo), hi)
        return t

    a = float(v[live].min()) - hi   # f(a) = N * hi >= 0
    b = float(v[live].max()) - lo   # f(b) = N * lo <= 0
    for _ in range(iters):
        mid = 0.5 * (a + b)
        if f(mid) > 0:
            a = mid
        else:
            b = mid
    lam = 0.5 * (a + b)
    return np.where(live, np.clip(v - lam, lo, hi), np.clip(v, lo, hi))


def compass_candidates(u, v_clip, h, counts, bounds):
    """The trial points of one round around the incumbent (u = log gains,
    v_clip = log c): for every coordinate d (the S gains, then the threshold)
    a step of +h, then -h.  A gain step is projected with project_log_gains; a
    threshold step is clamped to [log c_min, log c_max].  Returns the fp32
    gains [2(S+1), S] and thresholds [2(S+1)], the values that are evaluated
    (clamped to the bounds after exponentiation), and their log coordinates."""
    g_min, g_max, c_min, c_max = (float(b) for b in bounds)
    lo, hi = np.log(g_min), np.log(g_max)
    S = len(u)
    gam, clip, us, vs = [], [], [], []
    for d in range(S + 1):
        for sign in (1.0, -1.0):
            if d < S:
                w = np.array(u, dtype=np.float64)
                w[d] += sign * h
                w = project_log_gains(w, counts, lo, hi)
                vc = v_clip
            else:
                w = np.array(u, dtype=np.float64)
                vc = min(max(v_clip + sign * h, np.log(c_min)), np.log(c_max))
            gam.append(np.clip(np.exp(w).astype(F32), F32(g_min), F32(g_max)))
            clip.append(np.clip(F32(np.exp(vc)), F32(c_min), F32(c_max)))
            us.append(w)
            vs.append(vc)
    return np.stack(gam), np.array(clip, dtype=F32), np.stack(us), np.array(vs)


def calib_search(objective, counts, bounds, clip_init, log_step, rounds):
    """Compass search for Eq. (9)'s (gamma*, c*).  objective(gammas [C, S],
    clips [C]) -> float64 [C].  Starts from gamma = 1 (which meets every
    constraint) and c = clip_init clamped to [c_min, c_max], with step
    log_step.  Each round evaluates compass_candidates; the first candidate
    with the smallest objective replaces the incumbent if it is strictly
    better, else the step halves.  Returns (gamma fp32 [S], c fp32, L, step,
    trace); trace holds per round the candidates' objectives and the
    incumbent's before the round."""
    g_min, g_max, c_min, c_max = (float(b) for b in bounds)
    S = len(counts)
    u = np.zeros(S)
    gam = np.ones(S, dtype=F32)
    c = np.clip(F32(clip_init), F32(c_min), F32(c_max))
    vc = float(np.log(np.float64(c)))
    L = float(objective(gam[None, :], np.array([c], dtype=F32))[0])
    h = float(log_step)
    trace = []
    for _ in range(rounds):
        G, C, U, V = compass_candidates(u, vc, h, counts, bounds)
        obj = np.asarray(objective(G, C), dtype=np.float64)
        trace.append((L, obj))
        j = int(np.argmin(obj))
        if obj[j] < L:
            L, u, vc, gam, c = float(obj[j]), U[j], float(V[j]), G[j], C[j]
        else:
            h = 0.5 * h
    return gam, F32(c), L, h, trace



# ---------------------------------------------------------------- shared channel scaling, Eq. (7)
# Eq. (7) chooses the shared scaling D* by the reconstruction error of
# Q(X D^-1) Q(D W) against the full-precision X W, weighted per region
# (tau, s); the paper names neither a family for D nor an optimizer.  The
# reading here: the one-parameter family below, searched over a list of
# exponents; the activation quantizer of the objective is the per-token (8-bit)
# or per-64-group (4-bit) absmax quantizer with unit gains (Eq. (7) has none).

def smooth_scales(x_bits, w, alpha):
    """d_k = amax_i |x_ik|^alpha / amax_j |w_jk|^(1 - alpha), evaluated in
    float64 (alpha taken as the fp32 value given), clamped to [2^-6, 2^6] and
    rounded to fp32; a channel whose amax is 0 on either side gets d = 1.
    Also returns dinv = fp32(1 / d).  x_bits: bf16 [M, K]; w: fp32 [N, K]."""
    ax = np.abs(bf16_bits_to_f32(np.asarray(x_bits, np.uint16))).max(axis=0).astype(np.float64)
    aw = np.abs(np.asarray(w, F32)).max(axis=0).astype(np.float64)
    a = float(F32(alpha))
    d = np.ones(ax.shape, dtype=np.float64)
    for k in range(ax.size):
        if ax[k] > 0 and aw[k] > 0:
            d[k] = ax[k] ** a / aw[k] ** (1.0 - a)
    d = np.minimum(np.maximum(d, 2.0 ** -6), 2.0 ** 6).astype(F32)
    return d, (F32(1.0) / d).astype(F32)


def scaling_objective(x_bits, region, num_regions, region_weight, w, w_group, alphas, act_bits=8, ref=None):
    """Eq. (7) for each exponent of the family (smooth_scales):

        L(D) = sum_r weight_r / n_r * || Q(X_r D^-1) Q(D W) - X_r W ||_F^2

    over regions r (an id per row, e.g. step x stream; weight_r = pi_tau
    omega^D_{tau,s}).  Q(D W) is pack_weights(w, d); Q(X D^-1) Q(D W) is the
    fused linear with DYNAMIC ranges, unit gains and no bias at its float64
    value; X W is full_precision_linear.  Returns float64 [len(alphas)]."""
    if ref is None:
        ref = full_precision_linear(x_bits, w)
    region = np.asarray(region, np.int32)
    ones = np.ones((1, num_regions), dtype=F32)
    out = []
    for alpha in np.asarray(alphas, dtype=F32):
        d, dinv = smooth_scales(x_bits, w, alpha)
        pw = pack_weights(w, d, w_group)
        res = linear(x_bits, region, ones, 0, pw["codes"], pw["w_scale"], w_group, dinv=dinv, bias_bits=None,
                     range_mode=RANGE_DYNAMIC, act_bits=act_bits)
        out.append(weighted_stream_error(res["y64"], ref, region, num_regions, region_weight))
    return np.array(out, dtype=np.float64)
