"""Pins of the CPU oracle against what the paper and the mathematics fix
(CPU only).  Each test names the passage it checks.

None of these re-types the oracle's formulas: they use special cases with
closed-form answers, exact rational brute force on tiny shapes, bounds and
exact invariants."""
from fractions import Fraction

import numpy as np
import pytest

from oracle import sq_oracle as O
from paper_2609_39056_amd import synth

F32 = np.float32


def _bits(x):
    return O.f32_to_bf16_bits(np.asarray(x, dtype=F32))


def _layer(K=256, N=64, counts=(24, 4, 8), T=3, seed=5, **kw):
    return synth.make_layer(K=K, N=N, stream_counts=counts, T=T, seed=seed, **kw)


# ---------------------------------------------------------------- P1
@pytest.mark.parametrize("act_bits", [8, 4])
def test_identity_special_case(act_bits):
    """Eq. (1) with c = q_max, gamma = 1, D = I: Delta = 1 and the quantizer is
    the identity on integers in [-q_max, q_max]; Eq. (2) then gives
    Y = X (Q_W Delta_W) exactly."""
    qa = O.Q_MAX[act_bits]
    rng = np.random.default_rng(0)
    M, K, N, T = 5, 128, 16, 2
    xi = rng.integers(-qa, qa + 1, size=(M, K))
    x_bits = _bits(xi)
    gamma = np.ones((T, 3), F32)
    clip = np.full(T, qa, F32)
    t2s = rng.integers(0, 3, M).astype(np.int32)
    q = O.quantize_act(x_bits, t2s, gamma, 1, clip=clip, range_mode=O.RANGE_STATIC, act_bits=act_bits)
    assert np.array_equal(q["codes"].astype(np.int64), xi)
    if act_bits == 8:
        assert np.all(q["scale"] == 1.0)
    else:
        assert np.all(q["scale"] == 0x3C00)  # fp16 1.0
    w = (rng.standard_normal((N, K)) * 0.02).astype(F32)
    pw = O.pack_weights(w, None, 128)
    bias = _bits(rng.standard_normal(N) * 0.1)
    res = O.linear(x_bits, t2s, gamma, 1, pw["codes"], pw["w_scale"], 128, clip=clip,
                   bias_bits=bias, range_mode=O.RANGE_STATIC, act_bits=act_bits)
    ws = O.f16_bits_to_f32(pw["w_scale"])
    b = O.bf16_bits_to_f32(bias)
    for i in range(M):
        for j in range(N):
            exact = sum(Fraction(int(xi[i, k])) * int(pw["codes"][j, k]) * Fraction(float(ws[j, k // 128]))
                        for k in range(K)) + Fraction(float(b[j]))
            assert abs(float(exact) - res["y64"][i, j]) <= 1e-12 * (res["A"][i, j] + 1e-30)
            assert abs(float(exact) - float(res["y"][i, j])) <= 4e-7 * res["A"][i, j]


# ---------------------------------------------------------------- P2
@pytest.mark.parametrize("act_bits", [8, 4])
def test_dynamic_absmax_full_range(act_bits):
    """DYNAMIC with gamma = 1 and D = I is the textbook symmetric absmax
    quantizer: each non-zero row (A8) or 64-group (A4) uses the full code
    range, its largest element mapping to +-q_max."""
    L = _layer()
    g1 = np.ones_like(L.gamma)
    q = O.quantize_act(L.x_bits, L.tok2stream, g1, 0, act_bits=act_bits)
    qa = O.Q_MAX[act_bits]
    G = L.K if act_bits == 8 else 64
    codes = q["codes"].reshape(L.M, L.K // G, G).astype(np.int64)
    x = O.bf16_bits_to_f32(L.x_bits).reshape(L.M, L.K // G, G)
    nz = np.abs(x).max(axis=2) > 0
    assert np.all(np.abs(codes).max(axis=2)[nz] == qa)
    am = np.abs(x).argmax(axis=2)
    top = np.take_along_axis(codes, am[..., None], axis=2)[..., 0]
    top_x = np.take_along_axis(x, am[..., None], axis=2)[..., 0]
    assert np.all(top[nz] == np.sign(top_x[nz]) * qa)
    # the step is amax / q_max (to fp32, or fp16 for A4) and, with gamma = 1,
    # nothing is clipped: every element reconstructs within half a step
    amax = np.abs(x.astype(np.float64)).max(axis=2)
    tol = 2.0**-23 if act_bits == 8 else 2.0**-11
    assert np.all(np.abs(q["delta"] - amax / qa) <= tol * amax / qa)
    d = q["delta"].astype(np.float64)[:, :, None]
    assert np.all(np.abs(x - codes * d) <= d * (0.5 + 2.0**-14))


def test_dynamic_zero_row():
    """An all-zero row has no range: codes 0 and row scale 0."""
    x_bits = np.zeros((2, 128), np.uint16)
    x_bits[1, 5] = _bits([1.5])[0]
    for bits in (8, 4):
        q = O.quantize_act(x_bits, np.zeros(2, np.int32), np.ones((1, 1), F32), 0, act_bits=bits)
        assert np.all(q["codes"][0] == 0)
        if bits == 8:
            assert q["scale"][0] == 0.0 and q["scale"][1] > 0
        else:
            assert np.all(q["scale"][0] == 0)


# ---------------------------------------------------------------- P3
@pytest.mark.parametrize("act_bits,mode", [(8, 0), (8, 1), (4, 0), (4, 1)])
def test_roundtrip_bound_and_saturation(act_bits, mode):
    """Eq. (1): unclipped elements reconstruct within half a step; App. C.1:
    the effective threshold of stream s is c / gamma_s and every element
    beyond it saturates.  Round-half-to-even: |q| = q_max iff t > q_max - 1/2."""
    L = _layer(seed=11)
    qa = O.Q_MAX[act_bits]
    clip = L.clip * F32(0.5)  # force some clipping in STATIC mode
    q = O.quantize_act(L.x_bits, L.tok2stream, L.gamma, 1, dinv=L.dinv, clip=clip,
                       range_mode=mode, act_bits=act_bits)
    G = L.K if act_bits == 8 else 64
    xt = q["xt"].astype(np.float64).reshape(L.M, -1, G)
    codes = q["codes"].astype(np.float64).reshape(L.M, -1, G)
    delta = q["delta"].astype(np.float64)[:, :, None]
    g = q["g"].astype(np.float64)[:, None, None]
    c = (np.full_like(delta, clip[1]) if mode == 1 else np.abs(xt).max(axis=2, keepdims=True))
    t_exact = xt * g / np.where(delta > 0, delta, 1.0)
    inside = np.abs(t_exact) <= qa - 0.5 - 1e-4
    err = np.abs(xt - codes * delta / g)
    assert np.all(err[inside] <= (delta / g * (0.5 + 2.0**-14) + 0 * err)[inside])
    beyond = np.abs(xt) >= (c / g) * (1 + 2.0**-20)
    assert beyond.any() or mode == 0
    assert np.all(np.abs(codes[beyond & (delta > 0)]) == qa)
    # the computed t decides saturation exactly
    t = ((q["xt"].reshape(L.M, -1, G) * q["g"][:, None, None]).astype(F32)
         * np.where(np.isinf(1 / q["delta"]), 0, (F32(1) / q["delta"]))[:, :, None].astype(F32)).astype(F32)
    sat = np.abs(codes) == qa
    assert np.array_equal(sat, np.abs(t) > qa - 0.5)


# ---------------------------------------------------------------- P4
@pytest.mark.parametrize("act_bits", [8, 4])
def test_power_of_two_invariance(act_bits):
    """Scaling X by 2^e (DYNAMIC) keeps the codes and scales the step by 2^e
    exactly; scaling gamma and c by 2^e (STATIC) keeps codes and r."""
    L = _layer(seed=3)
    e = 3
    x2 = O.f32_to_bf16_bits(O.bf16_bits_to_f32(L.x_bits) * F32(2.0**e))
    a = O.quantize_act(L.x_bits, L.tok2stream, L.gamma, 0, dinv=L.dinv, act_bits=act_bits)
    b = O.quantize_act(x2, L.tok2stream, L.gamma, 0, dinv=L.dinv, act_bits=act_bits)
    assert np.array_equal(a["codes"], b["codes"])
    sa = a["scale"] if act_bits == 8 else O.f16_bits_to_f32(a["scale"])
    sb = b["scale"] if act_bits == 8 else O.f16_bits_to_f32(b["scale"])
    assert np.array_equal(sa * F32(2.0**e), sb)
    s1 = O.quantize_act(L.x_bits, L.tok2stream, L.gamma, 0, dinv=L.dinv, clip=L.clip,
                        range_mode=O.RANGE_STATIC, act_bits=act_bits)
    s2 = O.quantize_act(L.x_bits, L.tok2stream, L.gamma * F32(4), 0, dinv=L.dinv, clip=L.clip * F32(4),
                        range_mode=O.RANGE_STATIC, act_bits=act_bits)
    assert np.array_equal(s1["codes"], s2["codes"])
    if act_bits == 8:
        assert np.array_equal(s1["scale"], s2["scale"])


# ---------------------------------------------------------------- P5
@pytest.mark.parametrize("act_bits", [8, 4])
def test_permutation_equivariance(act_bits):
    """Every step is row-independent: permuting rows of X together with the
    token->stream map permutes Q_X, the scales and Y bit-exactly."""
    L = _layer(seed=7, N=32)
    pw = O.pack_weights(L.w, L.d, 128)
    perm = np.random.default_rng(0).permutation(L.M)
    kw = dict(dinv=L.dinv, bias_bits=L.bias_bits, act_bits=act_bits)
    a = O.linear(L.x_bits, L.tok2stream, L.gamma, 1, pw["codes"], pw["w_scale"], 128, **kw)
    b = O.linear(L.x_bits[perm], L.tok2stream[perm], L.gamma, 1, pw["codes"], pw["w_scale"], 128, **kw)
    assert np.array_equal(a["codes"][perm], b["codes"])
    assert np.array_equal(a["scale"][perm], b["scale"])
    assert np.array_equal(a["y"][perm], b["y"])


# ---------------------------------------------------------------- P6
@pytest.mark.parametrize("G", [64, 128, 256])
def test_block_acc_bruteforce(G):
    """INT32 accumulation (Sec. 4.4): Python-integer triple loop."""
    rng = np.random.default_rng(G)
    M, N, K = 3, 5, 256
    qx = rng.integers(-127, 128, size=(M, K)).astype(np.int8)
    qw = rng.integers(-8, 8, size=(N, K)).astype(np.int8)
    C = O.block_acc(qx, qw, G)
    assert C.shape == (K // G, M, N)
    for b in range(K // G):
        for i in range(M):
            for j in range(N):
                s = 0
                for k in range(b * G, (b + 1) * G):
                    s += int(qx[i, k]) * int(qw[j, k])
                assert C[b, i, j] == s


# ---------------------------------------------------------------- P7
@pytest.mark.parametrize("act_bits,w_group", [(8, 128), (8, 256), (4, 128), (4, 256)])
def test_dequantized_product_exact(act_bits, w_group):
    """Eq. (2) with per-element steps and the gamma^-1 of Eq. (8):
    Y_ij = gamma_s(i)^-1 sum_k (q_ik Delta_X,ik)(q_jk Delta_W,jk) + b_j, in exact
    rational arithmetic from the oracle's own codes and steps, against the
    oracle's block-wise epilogue (fp64 shadow to 1e-12, fp32 to the summation
    bound).  Catches wrong block / group indices, transposes and a dropped
    compensation."""
    L = _layer(K=256, N=6, counts=(3, 2, 2), seed=21)
    pw = O.pack_weights(L.w, L.d, w_group)
    res = O.linear(L.x_bits, L.tok2stream, L.gamma, 1, pw["codes"], pw["w_scale"], w_group,
                   dinv=L.dinv, bias_bits=L.bias_bits, act_bits=act_bits)
    ws = O.f16_bits_to_f32(pw["w_scale"])
    b = O.bf16_bits_to_f32(L.bias_bits)
    G_a = L.K if act_bits == 8 else 64
    # the stored per-row factors are fp32 roundings of Delta/gamma (A8) and
    # 1/gamma (A4): check that, then use the stored values exactly
    gam = L.gamma[1, L.tok2stream].astype(np.float64)
    if act_bits == 8:
        assert np.all(np.abs(res["scale"] - res["delta"][:, 0] / gam) <= 2.0**-24 * res["scale"])
    assert np.all(np.abs(res["kappa"] - 1 / gam) <= 2.0**-24 * res["kappa"])
    for i in range(L.M):
        for j in range(L.N):
            acc = Fraction(0)
            for k in range(L.K):
                if act_bits == 8:
                    dx = Fraction(float(res["scale"][i]))
                else:
                    dx = Fraction(float(res["delta"][i, k // G_a]))
                dw = Fraction(float(ws[j, k // w_group]))
                acc += int(res["codes"][i, k]) * dx * int(pw["codes"][j, k]) * dw
            if act_bits == 4:
                acc *= Fraction(float(res["kappa"][i]))
            exact = acc + Fraction(float(b[j]))
            A = res["A"][i, j]
            assert abs(float(exact) - res["y64"][i, j]) <= 1e-12 * A
            nb = L.K // res["G"]
            assert abs(float(exact) - float(res["y"][i, j])) <= (nb + 4) * 2.0**-24 * A


# ---------------------------------------------------------------- P8
def test_channel_scaling_cancels_in_full_precision():
    """Eq. (6): X D^-1 and D W cancel in full precision.  With the oracle's
    own fp32 X D^-1 and D W, the fp64 product equals X W up to the three fp32
    roundings per term.  A D applied along the wrong axis fails this."""
    L = _layer(K=256, N=48, seed=4)
    q = O.quantize_act(L.x_bits, L.tok2stream, L.gamma, 0, dinv=L.dinv)
    wf = (L.w * L.d[None, :]).astype(F32)
    pw = O.pack_weights(L.w, L.d, 128)
    # the oracle's folded weight is the one it quantizes: reconstruct it
    ws = O.f16_bits_to_f32(pw["w_scale"]).astype(np.float64)
    recon = pw["codes"].astype(np.float64) * np.repeat(ws, 128, axis=1)
    assert np.all(np.abs(recon - wf) <= np.repeat(ws, 128, axis=1) * (0.5 + 2.0**-14))
    y_fold = q["xt"].astype(np.float64) @ wf.astype(np.float64).T
    y_ref = O.full_precision_linear(L.x_bits, L.w)
    mag = np.abs(q["xt"].astype(np.float64)) @ np.abs(wf.astype(np.float64)).T
    assert np.all(np.abs(y_fold - y_ref) <= 4 * 2.0**-24 * mag)
    # and D must not be the identity here, else the check is vacuous
    assert np.abs(L.d - 1).max() > 0.5


# ---------------------------------------------------------------- P9
@pytest.mark.parametrize("act_bits", [8, 4])
def test_compensation_exact_and_effective(act_bits):
    """Eq. (8): the inverse gain compensates the input scaling.  (a) Scaling
    every gain and c by 2^e leaves Y bit-identical (STATIC).  (b) With a large
    threshold (no clipping) and gains drawn per stream, Y stays within the
    rounding bound of X D^-1 W^ whatever the gains; dropping gamma^-1 would
    scale each stream's output by gamma."""
    L = _layer(seed=9, N=32)
    pw = O.pack_weights(L.w, L.d, 128)
    kw = dict(dinv=L.dinv, bias_bits=None, range_mode=O.RANGE_STATIC, act_bits=act_bits)
    a = O.linear(L.x_bits, L.tok2stream, L.gamma, 2, pw["codes"], pw["w_scale"], 128, clip=L.clip, **kw)
    b = O.linear(L.x_bits, L.tok2stream, L.gamma * F32(0.25), 2, pw["codes"], pw["w_scale"], 128,
                 clip=L.clip * F32(0.25), **kw)
    assert np.array_equal(a["y"], b["y"])
    # (b) no clipping: c large enough for every stream's effective range
    xt = a["xt"].astype(np.float64)
    gam = np.array([[0.5, 2.0, 1.3]] * L.T, F32)
    big = F32(np.abs(xt).max() * float(gam.max()) * 1.01)
    r = O.linear(L.x_bits, L.tok2stream, gam, 0, pw["codes"], pw["w_scale"], 128,
                 clip=np.full(L.T, big, F32), **kw)
    ws = np.repeat(O.f16_bits_to_f32(pw["w_scale"]).astype(np.float64), 128, axis=1)
    what = pw["codes"].astype(np.float64) * ws
    target = xt @ what.T
    step = (r["delta"][:, 0].astype(np.float64) / r["g"].astype(np.float64))[:, None]
    bound = 0.5001 * step * np.abs(what).sum(axis=1)[None, :] + 1e-6 * np.abs(target)
    assert np.all(np.abs(r["y64"] - target) <= bound)


# ---------------------------------------------------------------- weights
@pytest.mark.parametrize("w_group", [128, 256])
def test_weight_quantizer(w_group):
    """Sec. 4.2 folding, then Eq. (1) for weights (k = 4, q_max = 7) per group:
    the fp16 step is amax/7 to fp16 precision, each group's largest element
    maps to +-7 and every element reconstructs within half a step."""
    L = _layer(K=512, N=40, seed=13)
    pw = O.pack_weights(L.w, L.d, w_group)
    wf = (L.w.astype(np.float64) * L.d.astype(np.float64)[None, :]).reshape(L.N, -1, w_group)
    ws = O.f16_bits_to_f32(pw["w_scale"]).astype(np.float64)
    amax = np.abs(wf).max(axis=2)
    assert np.all(np.abs(ws - amax / 7) <= 2.0**-11 * amax / 7 * 1.0001)
    codes = pw["codes"].reshape(L.N, -1, w_group).astype(np.float64)
    assert np.all(np.abs(codes).max(axis=2) == 7)
    assert np.all(np.abs(wf - codes * ws[:, :, None]) <= ws[:, :, None] * (0.5 + 2.0**-14) + 1e-12)
    assert np.array_equal(O.unpack_int4(pw["qw"]), pw["codes"])


def test_quantized_layer_is_close_to_full_precision():
    """Sanity of the whole chain on the 88-token 256x256 layer: W4A8 output
    stays close to the full-precision X W (normalized error of Eq. (3))."""
    L = synth.make_layer(**{k: v for k, v in synth.SMALL_LAYER.items() if k != "name"}, seed=0)
    pw = O.pack_weights(L.w, L.d, 128)
    r = O.linear(L.x_bits, L.tok2stream, L.gamma, 0, pw["codes"], pw["w_scale"], 128,
                 dinv=L.dinv, bias_bits=L.bias_bits)
    y_fp = O.full_precision_linear(L.x_bits, L.w, L.bias_bits)
    # undo the gain: with DYNAMIC ranges a gain > 1 clips, so compare the
    # rows whose gain is <= 1 (no clipping), where only rounding error remains
    ok = r["g"] <= 1.0
    eps = np.linalg.norm(r["y64"][ok] - y_fp[ok]) / np.linalg.norm(y_fp[ok])
    assert ok.any() and eps < 0.2


# ---------------------------------------------------------------- calibration objective, Eq. (9)
@pytest.mark.parametrize("act_bits", [8, 4])
def test_calib_objective_zero_on_representable_input(act_bits):
    """Sec. 4.3 Eq. (8)-(9): when every gamma_s x~ is a multiple of Delta =
    c / q_max inside [-c, c], Q reproduces it exactly and gamma_s^-1 undoes
    the gain, so the modulated output equals X~ W^ and the objective is 0
    (up to float64 summation order).  Gains are powers of two, so every
    scale involved is exact; a lost compensation, step or gain shows."""
    qa = O.Q_MAX[act_bits]
    rng = np.random.default_rng(11)
    M, K, N, S = 12, 256, 64, 3
    delta = 2.0 ** -4
    c = np.float32(qa * delta)
    gam = np.array([1.0, 2.0, 0.5], F32)
    t2s = (np.arange(M) % S).astype(np.int32)
    k = rng.integers(-qa, qa + 1, size=(M, K))
    x = (k * delta / gam[t2s][:, None]).astype(F32)       # gamma_s x = k Delta, exact in bf16
    x_bits = _bits(x)
    assert np.array_equal(O.bf16_bits_to_f32(x_bits), x)
    w = rng.standard_normal((N, K)).astype(F32) * 0.05
    pw = O.pack_weights(w, None, 128)
    ref = O.calib_reference(x_bits, pw["codes"], pw["w_scale"], 128)
    L = O.calib_objective(x_bits, t2s, S, pw["codes"], pw["w_scale"], 128, gam[None, :], [c], np.ones(S) / S,
                          act_bits=act_bits, ref=ref)
    assert L[0] <= 1e-24 * float((ref ** 2).mean())
    # the same input with the gains off: clipping and rounding errors appear
    L1 = O.calib_objective(x_bits, t2s, S, pw["codes"], pw["w_scale"], 128, np.ones((1, S), F32), [c],
                           np.ones(S) / S, act_bits=act_bits, ref=ref)
    assert L1[0] > 1e-6 * float((ref ** 2).mean())


def test_calib_objective_homogeneous():
    """Eq. (1), (9): scaling X and c by 2 leaves the codes unchanged and
    doubles both outputs exactly, so the objective grows by exactly 4."""
    L_ = _layer(K=256, N=64, counts=(20, 4, 8), seed=12)
    pw = O.pack_weights(L_.w, L_.d, 128)
    x2 = O.f32_to_bf16_bits(2 * O.bf16_bits_to_f32(L_.x_bits))
    g = np.array([[1.0, 1.5, 0.75], [0.9, 1.0, 1.25]], F32)
    c = np.array([3.0, 5.0], F32)
    om = np.array([0.5, 0.25, 0.25])
    a = O.calib_objective(L_.x_bits, L_.tok2stream, 3, pw["codes"], pw["w_scale"], 128, g, c, om, dinv=L_.dinv)
    b = O.calib_objective(x2, L_.tok2stream, 3, pw["codes"], pw["w_scale"], 128, g, 2 * c, om, dinv=L_.dinv)
    assert np.array_equal(b, 4 * a)


def test_calib_objective_streams_separate():
    """Eq. (9): stream t's gain only moves stream t's term: with all weight
    on stream 0, changing gamma_1 and gamma_2 leaves the objective unchanged,
    and with all weight on stream 1 changing gamma_1 moves it."""
    L_ = _layer(K=256, N=64, counts=(20, 6, 8), seed=13)
    pw = O.pack_weights(L_.w, L_.d, 128)
    g = np.array([[1.0, 1.0, 1.0], [1.0, 3.0, 0.3]], F32)
    c = np.array([4.0, 4.0], F32)
    on0 = O.calib_objective(L_.x_bits, L_.tok2stream, 3, pw["codes"], pw["w_scale"], 128, g, c, [1, 0, 0],
                            dinv=L_.dinv)
    on1 = O.calib_objective(L_.x_bits, L_.tok2stream, 3, pw["codes"], pw["w_scale"], 128, g, c, [0, 1, 0],
                            dinv=L_.dinv)
    assert on0[0] == on0[1] and on1[0] != on1[1]


# ---------------------------------------------------------------- constrained (gamma, c) search, Eq. (9)
def test_projection_closed_form_inside_bounds():
    """With no bound active the token-weighted projection onto
    sum_s n_s u_s = 0 subtracts the token-weighted mean: u = v - sum(n v) / sum(n)."""
    rng = np.random.default_rng(20)
    for S in (1, 2, 3, 9):
        n = rng.integers(1, 5000, S)
        v = rng.normal(0, 0.2, S)
        u = O.project_log_gains(v, n, -5.0, 5.0)
        assert np.allclose(u, v - (n * v).sum() / n.sum(), rtol=0, atol=1e-12)


def test_projection_matches_active_set_enumeration():
    """App. C.1 constraint set with bounds that bind: the projection equals
    the best feasible point over every active set (each coordinate free, at
    its lower or at its upper bound; the free ones then have the closed form
    v - mu), i.e. brute force on the convex problem min sum n (u - v)^2; a
    stream without tokens is only clamped."""
    import itertools
    rng = np.random.default_rng(21)
    lo, hi = np.log(0.5), np.log(2.0)
    for trial in range(8):
        S = 4
        n = rng.integers(1, 200, S).astype(float)
        v = rng.normal(0, 1.0, S)
        u = O.project_log_gains(v, n, lo, hi)
        assert np.all(u >= lo) and np.all(u <= hi)
        assert abs((n * u).sum()) <= 1e-9 * n.sum()
        best, best_u = np.inf, None
        for act in itertools.product((0, 1, 2), repeat=S):
            z = np.where(np.array(act) == 1, lo, hi).astype(float)
            free = np.array(act) == 0
            if free.any():
                mu = ((n * v)[free].sum() + (n * z)[~free].sum()) / n[free].sum()
                z[free] = v[free] - mu
            if abs((n * z).sum()) > 1e-9 * n.sum() or np.any(z < lo - 1e-12) or np.any(z > hi + 1e-12):
                continue
            val = float((n * (z - v) ** 2).sum())
            if val < best:
                best, best_u = val, z
        assert np.allclose(u, best_u, atol=1e-9)
    u = O.project_log_gains(np.array([3.0, 0.4, -0.2]), np.array([0, 10, 10]), lo, hi)
    assert u[0] == hi and abs(u[1] + u[2]) < 1e-12 and abs(u[1] - 0.3) < 1e-12
    u = O.project_log_gains(np.array([0.3, 0.4, -0.2]), np.array([0, 10, 10]), lo, hi)
    assert u[0] == 0.3 and abs(u[1] - 0.3) < 1e-12


def test_compass_search_finds_the_constrained_minimum_of_a_quadratic():
    """The search procedure on an objective with a known constrained
    minimizer: f = sum_s n_s (log gamma_s - a_s)^2 + (log c - b)^2, whose
    minimizer on the constraint set (bounds inactive) is log gamma =
    a - weighted mean of a, c = e^b."""
    n = np.array([4096, 32, 64])
    a = np.array([0.1, -0.4, 0.7])
    b = np.log(3.0)

    def f(G, C):
        return ((n[None, :] * (np.log(G.astype(np.float64)) - a[None, :]) ** 2).sum(1)
                + (np.log(C.astype(np.float64)) - b) ** 2)

    gam, c, L, h, trace = O.calib_search(f, n, (0.25, 4.0, 0.5, 20.0), 1.0, 0.5, 80)
    u_star = a - (n * a).sum() / n.sum()
    assert np.allclose(np.log(gam.astype(np.float64)), u_star, atol=2e-3)
    assert abs(np.log(float(c)) - b) < 2e-3
    assert abs((n * np.log(gam.astype(np.float64))).sum()) < 1e-3 * n.sum()
    # the incumbent's objective never rises
    inc = [t[0] for t in trace] + [L]
    assert all(x >= y for x, y in zip(inc, inc[1:]))


def test_calib_search_on_a_layer():
    """The search on Eq. (9) itself (three streams, uniform weights): every
    constraint holds at the result, the objective does not rise from the
    start (gamma = 1, c = clip_init), and the returned L is the objective of
    the returned point."""
    L_ = _layer(K=256, N=64, counts=(40, 6, 10), seed=22)
    pw = O.pack_weights(L_.w, L_.d, 128)
    n = np.bincount(L_.tok2stream, minlength=3)
    om = np.full(3, 1 / 3)
    ref = O.calib_reference(L_.x_bits, pw["codes"], pw["w_scale"], 128, L_.dinv)

    def f(G, C):
        return O.calib_objective(L_.x_bits, L_.tok2stream, 3, pw["codes"], pw["w_scale"], 128, G, C, om,
                                 dinv=L_.dinv, act_bits=4, ref=ref)

    bounds = (0.5, 2.0, 0.1, 50.0)
    gam, c, L, h, trace = O.calib_search(f, n, bounds, float(L_.clip[0]), 0.5, 10)
    assert np.all(gam >= F32(0.5)) and np.all(gam <= F32(2.0)) and F32(0.1) <= c <= F32(50.0)
    assert abs((n * np.log(gam.astype(np.float64))).sum()) < 1e-5 * n.sum()
    assert L <= trace[0][0]
    assert f(gam[None, :], np.array([c]))[0] == L


def test_calib_search_single_stream_keeps_unit_gain():
    """One stream: sum n log gamma = 0 forces gamma = 1 exactly (only the
    threshold moves)."""
    n = np.array([50])
    gam, c, L, h, _ = O.calib_search(lambda G, C: (np.log(C.astype(np.float64)) - 1.0) ** 2
                                     + (G[:, 0].astype(np.float64) - 3.0) ** 2, n, (0.5, 2.0, 0.1, 10.0), 1.0, 0.5, 30)
    assert gam[0] == F32(1.0) and abs(np.log(float(c)) - 1.0) < 1e-3


def test_calib_objective_token_mean_per_stream():
    """Eq. (9) divides each stream's squared error by its token count: the
    same calibration batch given twice (every row duplicated) leaves the
    objective unchanged, and so does doubling one stream's rows alone."""
    L_ = _layer(K=256, N=64, counts=(20, 6, 8), seed=14)
    pw = O.pack_weights(L_.w, L_.d, 128)
    g = np.array([[1.0, 1.5, 0.75], [0.8, 1.0, 1.3]], F32)
    c = np.array([4.0, 3.0], F32)
    om = np.array([0.5, 0.3, 0.2])

    def obj(xb, t2s):
        return O.calib_objective(xb, t2s, 3, pw["codes"], pw["w_scale"], 128, g, c, om, dinv=L_.dinv)

    base = obj(L_.x_bits, L_.tok2stream)
    twice = obj(np.concatenate([L_.x_bits, L_.x_bits]), np.concatenate([L_.tok2stream, L_.tok2stream]))
    assert np.allclose(twice, base, rtol=1e-12, atol=0)
    s1 = L_.tok2stream == 1
    more = obj(np.concatenate([L_.x_bits, L_.x_bits[s1]]), np.concatenate([L_.tok2stream, L_.tok2stream[s1]]))
    assert np.allclose(more, base, rtol=1e-12, atol=0)


def test_calib_objective_zero_with_channel_scaling():
    """The target of Eq. (9) is X D^-1 W^: with power-of-two D^-1 and inputs
    whose gamma_s x D^-1 are representable codes, the modulated output equals
    X D^-1 W^ exactly and the objective is 0; dropping D^-1 from either side
    would leave a nonzero error."""
    rng = np.random.default_rng(15)
    M, K, N, S = 12, 256, 64, 3
    delta = 2.0 ** -4
    c = np.float32(127 * delta)
    gam = np.array([1.0, 2.0, 0.5], F32)
    dinv = (2.0 ** rng.integers(-2, 3, K)).astype(F32)
    t2s = (np.arange(M) % S).astype(np.int32)
    k = rng.integers(-127, 128, size=(M, K))
    x = (k * delta / gam[t2s][:, None] / dinv[None, :]).astype(F32)
    x_bits = _bits(x)
    assert np.array_equal(O.bf16_bits_to_f32(x_bits), x)
    w = rng.standard_normal((N, K)).astype(F32) * 0.05
    pw = O.pack_weights(w, None, 128)
    ref = O.calib_reference(x_bits, pw["codes"], pw["w_scale"], 128, dinv)
    L = O.calib_objective(x_bits, t2s, S, pw["codes"], pw["w_scale"], 128, gam[None, :], [c], np.ones(S) / S,
                          dinv=dinv, ref=ref)
    assert L[0] <= 1e-24 * float((ref ** 2).mean())
    ref_nod = O.calib_reference(x_bits, pw["codes"], pw["w_scale"], 128)
    assert float(((ref - ref_nod) ** 2).mean()) > 1e-6 * float((ref ** 2).mean())


def test_compass_candidates_respect_the_bounds():
    """Every trial point of a round lies in the constraint set (App. C.1) in
    its log coordinates as well as in its evaluated fp32 values, also when the
    incumbent sits on a bound: a threshold step past c_max stays at log c_max."""
    n = np.array([100, 10, 0])
    bounds = (0.5, 2.0, 0.25, 4.0)
    u = np.array([np.log(2.0), -np.log(2.0) * 10 / 10, 0.0])
    u = O.project_log_gains(u, n, np.log(0.5), np.log(2.0))
    G, C, U, V = O.compass_candidates(u, np.log(4.0), 0.7, n, bounds)
    assert G.shape == (8, 3) and C.shape == (8,)
    assert np.all(U >= np.log(0.5) - 1e-15) and np.all(U <= np.log(2.0) + 1e-15)
    assert np.all(V >= np.log(0.25) - 1e-15) and np.all(V <= np.log(4.0) + 1e-15)
    assert np.all(G >= F32(0.5)) and np.all(G <= F32(2.0)) and np.all(C >= F32(0.25)) and np.all(C <= F32(4.0))
    assert np.all(np.abs((n * U).sum(axis=1)) <= 1e-9 * n.sum())
    # the threshold's +h step is clamped to the bound, its -h step moves down by h
    assert V[6] == np.log(4.0) and abs(V[7] - (np.log(4.0) - 0.7)) < 1e-15


# ---------------------------------------------------------------- shared channel scaling, Eq. (7)
def test_smooth_scales_closed_forms():
    """The family at its ends and middle: alpha = 1 gives d = amax|X| and
    alpha = 0 gives 1 / amax|W| exactly (within the clamp), alpha = 1/2 the
    square root of their ratio to within fp32 rounding; zero channels give 1."""
    rng = np.random.default_rng(30)
    K = 64
    x = (rng.standard_normal((16, K)) * 2.0 ** rng.integers(-3, 4, K)).astype(F32)
    x[:, 5] = 0.0
    x[:, 7] *= 400.0  # amax above 2^6: the clamp binds at alpha = 1
    xb = _bits(x)
    xf = O.bf16_bits_to_f32(xb).astype(np.float64)
    w = (rng.standard_normal((8, K)) * 0.05).astype(F32)
    w[:, 9] = 0.0
    ax, aw = np.abs(xf).max(0), np.abs(w.astype(np.float64)).max(0)
    clamp = lambda v: np.minimum(np.maximum(v, 2.0 ** -6), 2.0 ** 6)
    live = (ax > 0) & (aw > 0)
    d1, _ = O.smooth_scales(xb, w, 1.0)
    assert np.array_equal(d1[live], clamp(ax[live]).astype(F32))
    d0, _ = O.smooth_scales(xb, w, 0.0)
    assert np.array_equal(d0[live], clamp(1.0 / aw[live]).astype(F32))
    dh, dinv = O.smooth_scales(xb, w, 0.5)
    want = clamp(np.sqrt(ax[live] / aw[live]))
    assert np.all(np.abs(dh[live] - want) <= 2.0 ** -23 * want)
    assert dh[5] == 1.0 and dh[9] == 1.0 and d0[5] == 1.0 and d1[7] == 64.0
    assert np.array_equal(dinv, (F32(1.0) / dh).astype(F32))


@pytest.mark.parametrize("act_bits", [8, 4])
def test_scaling_objective_homogeneous(act_bits):
    """Eq. (7) with the family's ends: at alpha = 1 doubling X doubles d, so
    X D^-1 and the codes stay and only the weight steps double; at alpha = 0
    doubling W halves d, so D W stays and the activation steps double.  Either
    way both the quantized and the full-precision outputs double exactly and
    the objective grows by exactly 4."""
    L_ = _layer(K=256, N=64, counts=(20, 4, 8), seed=31)
    reg = L_.tok2stream
    om = np.array([0.5, 0.3, 0.2])
    # X scaled by 2^-5 (exact) so that d = amax|X| stays inside the clamp [2^-6, 2^6] when doubled
    x1 = O.f32_to_bf16_bits(O.bf16_bits_to_f32(L_.x_bits) * F32(2.0 ** -5))
    assert np.abs(O.bf16_bits_to_f32(x1)).max() < 32
    x2 = O.f32_to_bf16_bits(2 * O.bf16_bits_to_f32(x1))
    a = O.scaling_objective(x1, reg, 3, om, L_.w, 128, [1.0], act_bits=act_bits)
    b = O.scaling_objective(x2, reg, 3, om, L_.w, 128, [1.0], act_bits=act_bits)
    assert b[0] == 4 * a[0] and a[0] > 0
    assert 1 / np.abs(L_.w).max(0).min() < 32
    a0 = O.scaling_objective(L_.x_bits, reg, 3, om, L_.w, 128, [0.0], act_bits=act_bits)
    b0 = O.scaling_objective(L_.x_bits, reg, 3, om, 2 * L_.w, 128, [0.0], act_bits=act_bits)
    assert b0[0] == 4 * a0[0] and a0[0] > 0


def test_scaling_objective_regions_and_scaling_matter():
    """The region weights average per region (the batch given twice leaves
    the objective unchanged); D matters: the exponents give different
    objectives on a layer with outlier channels, and at alpha = 1/2 the
    objective is below that of D = I (alpha chosen so d = 1 is not in the
    family) for this outlier-heavy input."""
    L_ = _layer(K=256, N=64, counts=(30, 6, 10), seed=32)
    reg, om = L_.tok2stream, np.full(3, 1 / 3)
    al = [0.0, 0.5, 1.0]
    a = O.scaling_objective(L_.x_bits, reg, 3, om, L_.w, 128, al)
    b = O.scaling_objective(np.concatenate([L_.x_bits, L_.x_bits]), np.concatenate([reg, reg]), 3, om, L_.w, 128, al)
    assert np.allclose(a, b, rtol=1e-12, atol=0)
    assert len(set(a.tolist())) == 3
    pw = O.pack_weights(L_.w, None, 128)
    ones = np.ones((1, 3), F32)
    res = O.linear(L_.x_bits, reg, ones, 0, pw["codes"], pw["w_scale"], 128, bias_bits=None)
    plain = O.weighted_stream_error(res["y64"], O.full_precision_linear(L_.x_bits, L_.w), reg, 3, om)
    assert a[1] < plain
