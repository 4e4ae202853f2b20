"""The C ABI on the host (no GPU): the library loads, exports every entry point
include/sq.h declares, and rejects invalid arguments before launching
anything.  Every call below fails validation, so no kernel is enqueued and the
HIP runtime is never asked for a device."""
import ctypes
import os
import re

import pytest

from paper_2609_39056_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "sq.h")

OK, NULL, SHAPE, ALIGN, UNSUP, WS = 0, -1, -2, -3, -4, -5
A = 0x10000  # a fake, suitably aligned device address (never dereferenced)


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(B.LIB_PATH):
        from paper_2609_39056_amd import _build
        _build.build()
    return B.lib()


def declared_symbols():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(sq_[a-z0-9_]+)\s*\(", text)))


def test_header_symbols_exported(L):
    syms = declared_symbols()
    assert "sq_linear_w4a8" in syms and "sq_linear_w4a4" in syms and "sq_linear_unfused" in syms
    assert "sq_quantize_act" in syms
    for s in syms:
        assert hasattr(L, s), s
    assert set(syms) == set(B._SIGS), "binding and header disagree"


def test_status_strings(L):
    for code in (OK, NULL, SHAPE, ALIGN, UNSUP, WS, -6):
        assert B.status_string(code).startswith("SQ_")
    assert "unknown" in B.status_string(42)


def test_workspace_bytes(L):
    M, K, N = 4192, 2048, 8192
    fused8 = B.sq_workspace_bytes(B.SQ_VARIANT_FUSED, M, K, N, 8)
    fused4 = B.sq_workspace_bytes(B.SQ_VARIANT_FUSED, M, K, N, 4)
    assert fused8 >= M * K + 4 * M and fused8 % 256 == 0
    assert fused4 >= M * K // 2 + 2 * M * (K // 64)
    unf = B.sq_workspace_bytes(B.SQ_VARIANT_UNFUSED, M, K, N, 8)
    assert unf >= 8 * M * K + 12 * M * N
    assert B.sq_workspace_bytes(B.SQ_VARIANT_FUSED, 0, K, N, 8) == 0
    assert B.sq_workspace_bytes(B.SQ_VARIANT_FUSED, M, 100, N, 8) == 0
    assert B.sq_workspace_bytes(B.SQ_VARIANT_FUSED, M, K, 100, 8) == 0
    assert B.sq_workspace_bytes(B.SQ_VARIANT_FUSED, M, K, N, 5) == 0
    assert B.sq_workspace_bytes(7, M, K, N, 8) == 0
    # GEMM scratch (split-K partial sums): at least 256 bytes, 256-aligned, and
    # included in the fused workspace
    g8 = B.sq_workspace_bytes(B.SQ_VARIANT_GEMM, M, K, N, 8)
    assert g8 >= 256 and g8 % 256 == 0
    assert fused8 >= M * K + 4 * M + g8
    assert B.sq_workspace_bytes(B.SQ_VARIANT_GEMM, 88, 256, 256, 8) == 256  # 2 stages: never split
    assert B.sq_workspace_bytes(B.SQ_VARIANT_GEMM, M, K, 100, 8) == 0


def act(**kw):
    d = dict(tok2stream=A, gamma=A, clip=A, dinv=None, num_streams=3, num_steps=2, step=0,
             range_mode=0, act_bits=8)
    d.update(kw)
    return B.sq_act_params(**d)


def wt(**kw):
    d = dict(qw=A, w_scale=A, bias=None, N=256, K=256, w_group=128)
    d.update(kw)
    return B.sq_weight(**d)


def quant(L, x=A, M=88, K=256, a=None, qx=A, sc=A):
    a = act() if a is None else a
    return L.sq_quantize_act(x, M, K, ctypes.byref(a) if a is not False else None, qx, sc, None)


@pytest.mark.parametrize("kw,code", [
    (dict(x=None), NULL), (dict(qx=None), NULL), (dict(sc=None), NULL), (dict(a=False), NULL),
    (dict(M=0), SHAPE), (dict(M=1 << 25), SHAPE), (dict(K=100), SHAPE), (dict(K=64), SHAPE),
    (dict(K=65536), SHAPE), (dict(x=A + 2), ALIGN), (dict(qx=A + 8), ALIGN), (dict(sc=A + 2), ALIGN),
])
def test_quantize_rejects(L, kw, code):
    assert quant(L, **kw) == code


@pytest.mark.parametrize("akw,code", [
    (dict(tok2stream=None), NULL), (dict(gamma=None), NULL), (dict(act_bits=5), UNSUP),
    (dict(range_mode=2), UNSUP), (dict(range_mode=1, clip=None), NULL), (dict(step=2), SHAPE),
    (dict(step=-1), SHAPE), (dict(num_streams=0), SHAPE), (dict(num_steps=0), SHAPE),
    (dict(dinv=A + 4), ALIGN), (dict(gamma=A + 1), ALIGN),
])
def test_act_params_rejected(L, akw, code):
    assert quant(L, a=act(**akw)) == code


def lin(L, fn="sq_linear_w4a8", x=A, M=88, a=None, w=None, y=A, out=0, ws=A, nbytes=1 << 30):
    a = act() if a is None else a
    w = wt() if w is None else w
    return getattr(L, fn)(x, M, ctypes.byref(a), ctypes.byref(w), y, out, ws, nbytes, None)


@pytest.mark.parametrize("fn", ["sq_linear_w4a8", "sq_linear_w4a4", "sq_linear_unfused"])
@pytest.mark.parametrize("kw,code", [
    (dict(x=None), NULL), (dict(y=None), NULL), (dict(ws=None), NULL), (dict(M=0), SHAPE),
    (dict(out=3), UNSUP), (dict(y=A + 4), ALIGN), (dict(ws=A + 8), ALIGN), (dict(nbytes=16), WS),
    (dict(w=wt(N=100)), SHAPE), (dict(w=wt(K=200)), SHAPE), (dict(w=wt(w_group=64)), UNSUP),
    (dict(w=wt(K=384, w_group=256)), UNSUP), (dict(w=wt(qw=None)), NULL), (dict(w=wt(w_scale=None)), NULL),
    (dict(w=wt(qw=A + 4)), ALIGN), (dict(w=wt(w_scale=A + 2)), ALIGN),
])
def test_linear_rejects(L, fn, kw, code):
    if fn == "sq_linear_w4a4":
        kw = dict(kw)
        kw.setdefault("a", act(act_bits=4))
    assert lin(L, fn=fn, **kw) == code


def test_linear_bits_mismatch(L):
    assert lin(L, "sq_linear_w4a8", a=act(act_bits=4)) == UNSUP
    assert lin(L, "sq_linear_w4a4", a=act(act_bits=8)) == UNSUP


def test_gemm_and_pack_reject(L):
    w = wt()
    assert L.sq_gemm_w4a8(None, A, 88, ctypes.byref(w), A, 0, None, 0, None) == NULL
    assert L.sq_gemm_w4a8(A, A, 0, ctypes.byref(w), A, 0, None, 0, None) == SHAPE
    assert L.sq_gemm_w4a8(A, A, 88, ctypes.byref(w), A, 0, A + 8, 1 << 20, None) == ALIGN
    a4 = act(act_bits=4)
    assert L.sq_gemm_w4a4(A, A, 88, ctypes.byref(act()), ctypes.byref(w), A, 0, None, 0, None) == UNSUP
    assert L.sq_gemm_w4a4(A, A + 2, 88, ctypes.byref(a4), ctypes.byref(w), A, 0, None, 0, None) == ALIGN
    assert L.sq_gemm_w4a4(A, A, 88, ctypes.byref(a4), ctypes.byref(w), A, 0, A + 4, 1 << 20, None) == ALIGN
    assert L.sq_pack_weights(A, None, 256, 256, 96, A, A, None) == UNSUP
    assert L.sq_pack_weights(A, None, 100, 256, 128, A, A, None) == SHAPE
    assert L.sq_pack_weights(None, None, 256, 256, 128, A, A, None) == NULL
    assert L.sq_pack_weights(A + 4, None, 256, 256, 128, A, A, None) == ALIGN
    assert L.sq_debug_block_acc_i32(A, 88, 6, ctypes.byref(w), A, None) == UNSUP
    assert L.sq_debug_block_acc_i32(None, 88, 8, ctypes.byref(w), A, None) == NULL


def test_binding_loads_only_the_built_library():
    assert B.LIB_PATH.endswith(os.path.join("paper_2609_39056_amd", "lib", "libsq.so"))


def test_mfma_probe_checks(L):
    """The matrix-core probe validates before launching (no GPU needed)."""
    n = L.sq_probe_mfma_i8_sink_bytes()
    assert n > 0 and n % 1024 == 0
    A = ctypes.c_void_p(1 << 20)  # never dereferenced: every call below fails validation
    for shape in (32, 16):
        assert L.sq_probe_mfma_i8(shape, 10, 1, 0, None, n, None) == NULL
        assert L.sq_probe_mfma_i8(shape, 0, 1, 0, A, n, None) == SHAPE
        assert L.sq_probe_mfma_i8(shape, (1 << 24) + 1, 1, 0, A, n, None) == SHAPE
        assert L.sq_probe_mfma_i8(shape, 10, 1, 0, A, n - 4, None) == WS
        assert L.sq_probe_mfma_i8(shape, 10, 1, 0, ctypes.c_void_p((1 << 20) + 2), n, None) == ALIGN
    for shape in (0, 8, 64):
        assert L.sq_probe_mfma_i8(shape, 10, 1, 0, A, n, None) == UNSUP
    for fmt in (8, 6):
        assert L.sq_probe_mfma_f8f6(fmt, 10, 1, 0, None, n, None) == NULL
        assert L.sq_probe_mfma_f8f6(fmt, 0, 1, 0, A, n, None) == SHAPE
        assert L.sq_probe_mfma_f8f6(fmt, (1 << 24) + 1, 1, 0, A, n, None) == SHAPE
        assert L.sq_probe_mfma_f8f6(fmt, 10, 1, 0, A, n - 4, None) == WS
        assert L.sq_probe_mfma_f8f6(fmt, 10, 1, 0, ctypes.c_void_p((1 << 20) + 2), n, None) == ALIGN
    for fmt in (0, 4, 16):
        assert L.sq_probe_mfma_f8f6(fmt, 10, 1, 0, A, n, None) == UNSUP


def calib(L, x=A, M=88, t2s=A, S=3, dinv=None, bits=8, w=None, ref=A, C=4, g=A, c=A, om=A, obj=A, ws=A,
          nbytes=1 << 30):
    w = wt() if w is None else w
    return L.sq_calib_objective(x, M, t2s, S, dinv, bits, ctypes.byref(w), ref, C, g, c, om, obj, ws, nbytes, None)


@pytest.mark.parametrize("kw,code", [
    (dict(x=None), NULL), (dict(t2s=None), NULL), (dict(ref=None), NULL), (dict(g=None), NULL),
    (dict(c=None), NULL), (dict(om=None), NULL), (dict(obj=None), NULL), (dict(ws=None), NULL),
    (dict(bits=5), UNSUP), (dict(M=0), SHAPE), (dict(S=0), SHAPE), (dict(S=4097), SHAPE), (dict(C=0), SHAPE),
    (dict(C=(1 << 16) + 1), SHAPE), (dict(x=A + 2), ALIGN), (dict(ref=A + 8), ALIGN), (dict(om=A + 4), ALIGN),
    (dict(obj=A + 4), ALIGN), (dict(g=A + 2), ALIGN), (dict(dinv=A + 4), ALIGN), (dict(ws=A + 8), ALIGN),
    (dict(nbytes=1024), WS), (dict(w=wt(N=100)), SHAPE), (dict(w=wt(qw=None)), NULL),
])
def test_calib_objective_rejects(L, kw, code):
    assert calib(L, **kw) == code


def test_calib_reference_rejects_and_sizes(L):
    w = wt()
    assert L.sq_calib_reference(None, 88, None, ctypes.byref(w), A, None) == NULL
    assert L.sq_calib_reference(A, 88, None, ctypes.byref(w), None, None) == NULL
    assert L.sq_calib_reference(A, 0, None, ctypes.byref(w), A, None) == SHAPE
    assert L.sq_calib_reference(A, 88, None, ctypes.byref(wt(K=200)), A, None) == SHAPE
    assert L.sq_calib_reference(A + 2, 88, None, ctypes.byref(w), A, None) == ALIGN
    assert L.sq_calib_reference(A, 88, A + 4, ctypes.byref(w), A, None) == ALIGN
    assert L.sq_calib_reference(A, 88, None, ctypes.byref(w), A + 8, None) == ALIGN
    M, K, N = 1000, 2048, 4096
    for bits in (8, 4):
        n = B.sq_calib_workspace_bytes(M, K, N, bits, 3)
        assert n % 256 == 0
        assert n >= B.sq_workspace_bytes(B.SQ_VARIANT_FUSED, M, K, N, bits) + 4 * M * N + 8 * M + 12
    assert B.sq_calib_workspace_bytes(M, K, N, 8, 0) == 0
    assert B.sq_calib_workspace_bytes(M, K, N, 8, 4097) == 0
    assert B.sq_calib_workspace_bytes(M, K, 100, 8, 3) == 0
    assert B.sq_calib_workspace_bytes(M, K, N, 6, 3) == 0


def search(L, x=A, M=88, t2s=A, S=3, dinv=None, bits=8, w=None, ref=A, om=A, p=None, g=A, c=A, obj=A, ws=A,
           nbytes=1 << 30):
    w = wt() if w is None else w
    if p is None:
        p = B.sq_calib_search_params(0.5, 2.0, 0.1, 10.0, 1.0, 0.5, 4)
    return L.sq_calib_search(x, M, t2s, S, dinv, bits, ctypes.byref(w), ref, om, ctypes.byref(p) if p else None,
                             g, c, obj, ws, nbytes, None)


def _sp(**kw):
    d = dict(gamma_min=0.5, gamma_max=2.0, clip_min=0.1, clip_max=10.0, clip_init=1.0, log_step=0.5, rounds=4)
    d.update(kw)
    return B.sq_calib_search_params(**d)


@pytest.mark.parametrize("kw,code", [
    (dict(x=None), NULL), (dict(t2s=None), NULL), (dict(ref=None), NULL), (dict(om=None), NULL), (dict(p=False), NULL),
    (dict(g=None), NULL), (dict(c=None), NULL), (dict(obj=None), NULL), (dict(ws=None), NULL), (dict(bits=6), UNSUP),
    (dict(M=0), SHAPE), (dict(S=0), SHAPE), (dict(S=65), SHAPE), (dict(p=_sp(rounds=-1)), SHAPE),
    (dict(p=_sp(rounds=1025)), SHAPE), (dict(p=_sp(gamma_min=0.0)), UNSUP), (dict(p=_sp(gamma_min=1.5)), UNSUP),
    (dict(p=_sp(gamma_max=0.9)), UNSUP), (dict(p=_sp(clip_min=0.0)), UNSUP), (dict(p=_sp(clip_max=0.05)), UNSUP),
    (dict(p=_sp(log_step=0.0)), UNSUP), (dict(p=_sp(log_step=65.0)), UNSUP), (dict(p=_sp(clip_init=float("inf"))), UNSUP),
    (dict(p=_sp(gamma_max=float("nan"))), UNSUP), (dict(x=A + 2), ALIGN), (dict(ref=A + 8), ALIGN),
    (dict(om=A + 4), ALIGN), (dict(g=A + 2), ALIGN), (dict(obj=A + 4), ALIGN), (dict(nbytes=4096), WS),
    (dict(w=wt(K=200)), SHAPE),
])
def test_calib_search_rejects(L, kw, code):
    assert search(L, **kw) == code


def test_calib_search_workspace(L):
    M, K, N = 1000, 2048, 4096
    for S in (1, 3, 64):
        n = B.sq_calib_search_workspace_bytes(M, K, N, 8, S)
        assert n > B.sq_calib_workspace_bytes(M, K, N, 8, S) and n % 256 == 0
    assert B.sq_calib_search_workspace_bytes(M, K, N, 8, 65) == 0
    assert B.sq_calib_search_workspace_bytes(M, K, N, 8, 0) == 0


def test_scaling_entry_points_reject(L):
    """Eq. (7) entry points validate before launching."""
    F = ctypes.c_float
    assert L.sq_calib_fp_reference(None, 88, A, 256, 256, A, None) == NULL
    assert L.sq_calib_fp_reference(A, 0, A, 256, 256, A, None) == SHAPE
    assert L.sq_calib_fp_reference(A, 88, A, 100, 256, A, None) == SHAPE
    assert L.sq_calib_fp_reference(A, 88, A + 4, 256, 256, A, None) == ALIGN
    assert L.sq_smooth_scales(A, 88, A, 256, 256, F(0.5), None, A + 1024, None) == NULL
    assert L.sq_smooth_scales(A, 88, A, 0, 256, F(0.5), A, A + 1024, None) == SHAPE
    assert L.sq_smooth_scales(A, 88, A, 256, 200, F(0.5), A, A + 1024, None) == SHAPE
    assert L.sq_smooth_scales(A, 88, A, 256, 256, F(float("nan")), A, A + 1024, None) == UNSUP
    assert L.sq_smooth_scales(A, 88, A, 256, 256, F(0.5), A, A, None) == UNSUP
    assert L.sq_smooth_scales(A + 2, 88, A, 256, 256, F(0.5), A, A + 1024, None) == ALIGN
    assert B.sq_calib_scaling_workspace_bytes(1000, 2048, 4096, 128, 8, 6) > B.sq_calib_workspace_bytes(1000, 2048,
                                                                                                        4096, 8, 6)
    assert B.sq_calib_scaling_workspace_bytes(1000, 2048, 4096, 96, 8, 6) == 0
    assert B.sq_calib_scaling_workspace_bytes(1000, 2048, 4096, 128, 8, 0) == 0
    al = (F * 3)(0.0, 0.5, 1.0)
    bad = (F * 2)(0.5, float("inf"))

    def so(x=A, M=88, reg=A, R=3, rw=A, w=A, N=256, K=256, G=128, bits=8, ref=A, n=3, alphas=al, obj=A, ws=A,
           nbytes=1 << 30):
        return L.sq_calib_scaling_objective(x, M, reg, R, rw, w, N, K, G, bits, ref, n, alphas, obj, ws, nbytes, None)

    for kw, code in [(dict(x=None), NULL), (dict(alphas=None), NULL), (dict(obj=None), NULL), (dict(bits=6), UNSUP),
                     (dict(M=0), SHAPE), (dict(R=0), SHAPE), (dict(R=4097), SHAPE), (dict(n=0), SHAPE),
                     (dict(G=96), UNSUP), (dict(alphas=bad, n=2), UNSUP), (dict(ref=A + 8), ALIGN),
                     (dict(rw=A + 4), ALIGN), (dict(nbytes=4096), WS), (dict(N=100), SHAPE)]:
        assert so(**kw) == code, kw


def test_static1_rejects(L):
    """The single-kernel STATIC linear validates before launching: it needs
    STATIC 8-bit ranges, at most 128 tokens and weight groups of 128 or K."""
    st = dict(range_mode=1)

    def s1(x=A, M=88, a=None, w=None, y=A, out=0, ws=None, nbytes=0):
        a = act(**st) if a is None else a
        w = wt() if w is None else w
        return L.sq_linear_w4a8_static1(x, M, ctypes.byref(a), ctypes.byref(w), y, out, ws, nbytes, None)

    assert s1(x=None) == NULL
    assert s1(y=None) == NULL
    assert s1(a=act()) == UNSUP                       # DYNAMIC ranges
    assert s1(a=act(range_mode=1, act_bits=4)) == UNSUP
    assert s1(a=act(range_mode=1, clip=None)) == NULL
    assert s1(M=129) == UNSUP                         # more than 128 tokens
    assert s1(M=0) == SHAPE
    assert s1(w=wt(K=512, w_group=256)) == UNSUP      # neither 128 nor K
    assert s1(out=3) == UNSUP
    assert s1(x=A + 2) == ALIGN
    assert s1(ws=A + 8, nbytes=1 << 20) == ALIGN


def test_gelu_quant_rejects(L):
    """The up projection with the GELU epilogue validates before launching:
    8-bit activations, 128-wide weight groups or one step per channel, and a
    STATIC 8-bit quantizer for the next layer, whose K is this layer's N."""
    big = 1 << 30

    def gq(x=A, M=300, a=None, w=None, an=None, qn=A, rn=A, ws=A, nbytes=big):
        a = act() if a is None else a
        w = wt() if w is None else w
        an = act(range_mode=1) if an is None else an
        return L.sq_linear_w4a8_gelu_quant(x, M, ctypes.byref(a), ctypes.byref(w), ctypes.byref(an), qn, rn, ws,
                                           nbytes, None)

    assert gq(x=None) == NULL
    assert gq(qn=None) == NULL
    assert gq(rn=None) == NULL
    assert gq(ws=None) == NULL
    assert gq(an=act()) == UNSUP                            # next layer DYNAMIC
    assert gq(an=act(range_mode=1, act_bits=4)) == UNSUP
    assert gq(an=act(range_mode=1, clip=None)) == NULL
    assert gq(a=act(act_bits=4)) == UNSUP
    assert gq(M=100, w=wt(K=512, w_group=256)) == UNSUP     # few tokens: groups of 128 or one step per channel
    assert gq(M=0) == SHAPE
    assert gq(w=wt(K=512, w_group=256)) == UNSUP
    assert gq(w=wt(N=192)) == SHAPE                         # next layer's K must be a multiple of 128
    assert gq(x=A + 2) == ALIGN
    assert gq(qn=A + 2) == ALIGN
    assert gq(rn=A + 2) == ALIGN
    assert gq(ws=A + 8) == ALIGN
    assert gq(an=act(range_mode=1, dinv=A + 4)) == ALIGN
    assert gq(nbytes=1024) == WS


def test_gelu_quant4_rejects(L):
    """The W4A4 up projection with the GELU epilogue: 4-bit activations for
    this layer and the next (STATIC), kc required for more than 128 tokens
    (the fp8 form), alignments, the workspace size."""
    big = 1 << 30

    def gq(x=A, M=300, a=None, w=None, an=None, qn=A, sn=A, kn=A, ws=A, nbytes=big):
        a = act(act_bits=4) if a is None else a
        w = wt() if w is None else w
        an = act(range_mode=1, act_bits=4) if an is None else an
        return L.sq_linear_w4a4_gelu_quant(x, M, ctypes.byref(a), ctypes.byref(w), ctypes.byref(an), qn, sn, kn, ws,
                                           nbytes, None)

    assert gq(x=None) == NULL
    assert gq(qn=None) == NULL
    assert gq(sn=None) == NULL
    assert gq(ws=None) == NULL
    assert gq(kn=None) == NULL                              # more than 128 tokens: the fp8 form needs kc
    assert gq(an=act(act_bits=4)) == UNSUP                  # next layer DYNAMIC
    assert gq(an=act(range_mode=1, act_bits=8)) == UNSUP
    assert gq(a=act(act_bits=8)) == UNSUP
    assert gq(an=act(range_mode=1, act_bits=4, clip=None)) == NULL
    assert gq(M=0) == SHAPE
    assert gq(w=wt(N=192)) == SHAPE                         # next layer's K must be a multiple of 128
    assert gq(x=A + 2) == ALIGN
    assert gq(qn=A + 2) == ALIGN
    assert gq(sn=A + 2) == ALIGN                            # fp32 steps
    assert gq(kn=A + 2) == ALIGN
    assert gq(M=100, kn=None, sn=A + 1) == ALIGN            # at most 128 tokens: fp16 steps, kc unused
    assert gq(ws=A + 8) == ALIGN
    assert gq(an=act(range_mode=1, act_bits=4, dinv=A + 4)) == ALIGN
    assert gq(nbytes=1024) == WS


def test_gemm_w4a4_fp8_rejects(L):
    """The 4-bit GEMM on fp8 code bytes: more than 128 tokens only (the packed
    form is sq_gemm_w4a4's), 4-bit activations, alignments."""
    def g8(qx=A, sg=A, kc=A, M=300, a=None, w=None, y=A, out=1, ws=None, nbytes=0):
        a = act(act_bits=4) if a is None else a
        w = wt() if w is None else w
        return L.sq_gemm_w4a4_fp8(qx, sg, kc, M, ctypes.byref(a), ctypes.byref(w), y, out, ws, nbytes, None)

    assert g8(qx=None) == NULL
    assert g8(sg=None) == NULL
    assert g8(kc=None) == NULL
    assert g8(y=None) == NULL
    assert g8(M=100) == UNSUP                               # few tokens: packed codes, sq_gemm_w4a4
    assert g8(a=act(act_bits=8)) == UNSUP
    assert g8(out=3) == UNSUP
    assert g8(M=0) == SHAPE
    assert g8(qx=A + 8) == ALIGN
    assert g8(sg=A + 2) == ALIGN
    assert g8(kc=A + 2) == ALIGN
    assert g8(y=A + 8) == ALIGN
    assert g8(ws=A + 8, nbytes=1 << 20) == ALIGN


def test_gelu_bf16_rejects(L):
    assert L.sq_gelu_bf16(None, 8, A, None) == NULL
    assert L.sq_gelu_bf16(A, 8, None, None) == NULL
    assert L.sq_gelu_bf16(A + 2, 8, A, None) == ALIGN
    assert L.sq_gelu_bf16(A, 8, A + 2, None) == ALIGN
    assert L.sq_gelu_bf16(None, 0, None, None) == OK        # nothing to do: no launch


def test_header_is_c_and_links(L, tmp_path):
    """include/sq.h compiles as C11 (-Wall -Werror) and a C program links
    libsq.so and calls two host-only entry points: the boundary is usable
    from C, not only through the Python binding."""
    import shutil
    import subprocess

    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    src = tmp_path / "use_sq.c"
    src.write_text(
        "#include <stdio.h>\n#include \"sq.h\"\n"
        "int main(void) {\n"
        "  size_t b = sq_workspace_bytes(SQ_VARIANT_FUSED, 300, 2048, 1024, 8);\n"
        "  printf(\"%s %zu\\n\", sq_status_string(SQ_ERR_SHAPE), b);\n"
        "  return b > 0 ? 0 : 1;\n}\n")
    libdir = os.path.dirname(B.LIB_PATH)
    exe = tmp_path / "use_sq"
    r = subprocess.run([cc, "-std=c11", "-Wall", "-Werror", "-D__HIP_PLATFORM_AMD__", f"-I{ROOT}/include",
                        "-I/opt/rocm/include", str(src), f"-L{libdir}", "-lsq", f"-Wl,-rpath,{libdir}",
                        "-o", str(exe)], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=60)
    assert r.returncode == 0, r.stderr
    msg, nbytes = r.stdout.rsplit(" ", 1)
    assert msg == B.status_string(SHAPE)
    assert int(nbytes) == B.sq_workspace_bytes(B.SQ_VARIANT_FUSED, 300, 2048, 1024, 8)
