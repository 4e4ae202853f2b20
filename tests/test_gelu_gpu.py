"""Producer-side fusion of the MLP chain (up projection -> GELU -> down
projection) and the bf16 GELU, through the C ABI, against the oracle.

The DiT block keeps GELU in bf16 between the two projections (App. D); the
up projection's GELU epilogue rounds Y to bf16, evaluates GELU with a fixed
fp32 sequence, rounds to bf16 and applies the down projection's STATIC 8-bit
quantizer (Eq. 1, 6, 8).  Bars:

* sq_gelu_bf16 equals the oracle's bf16 GELU on every one of the 65536 bf16
  bit patterns (NaN outputs compared as NaN);
* the fused chain's codes and row scales equal, bit for bit, those of the
  unfused GPU chain (sq_linear_w4a8 to bf16, sq_gelu_bf16, sq_quantize_act);
* row scales r equal the oracle's bit for bit (they depend on the step's
  threshold and the row's gain only);
* with inputs that make the up projection's fp32 output exact (integer
  activations, power-of-two steps; see test_exact_accum_gpu) the codes equal
  the oracle's chain bit for bit;
* with general inputs the up projection's bf16 output may differ from the
  oracle's by one ulp where its fp32 value sits next to a rounding boundary
  (summation order); wherever it does not, the codes are equal, and where it
  does they differ by at most 2 (one bf16 ulp of GELU's input moves the
  GELU output by at most about 1.13 ulp, then one more ulp from its own
  rounding, at most 127 * 2^-8 * 2.13 < 2 code steps).
"""
import numpy as np
import pytest
import torch

from gpu_util import act_params, bits16, expected_kc, f32_to_dev, i32_to_dev, oracle_weight, u16_to_dev
from oracle import sq_oracle as O
from paper_2609_39056_amd import binding as B
from paper_2609_39056_amd import synth
from test_exact_accum_gpu import ExactLayer, tile_rows

pytestmark = pytest.mark.gpu

T = 10


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.lib()


def same_bf16(got, want):
    """Bitwise equality of bf16 patterns, any NaN equal to any NaN."""
    gn = ((got & 0x7F80) == 0x7F80) & ((got & 0x7F) != 0)
    wn = ((want & 0x7F80) == 0x7F80) & ((want & 0x7F) != 0)
    return (gn & wn) | (~gn & ~wn & (got == want))


@pytest.mark.parametrize("n", [65536, 65531, 7, 0])
@pytest.mark.parametrize("in_place", [False, True])
def test_gelu_bf16_all_patterns(n, in_place):
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)[:n]
    want = O.gelu_bf16(bits)
    x = u16_to_dev(bits, torch.bfloat16) if n else torch.empty(0, dtype=torch.bfloat16, device="cuda")
    y = x if in_place else torch.full_like(x, float("nan"))
    B.sq_gelu_bf16(x, y)
    got = bits16(y) if n else np.zeros(0, np.uint16)
    ok = same_bf16(got, want)
    assert ok.all(), f"{(~ok).sum()} mismatches, first at input {bits[~ok][:5]}"


class DownParams:
    """The down projection's quantizer: gains [T, S], D^-1 [N_up] (or None),
    per-step thresholds [T].  Thresholds cover the 99.9th percentile of
    |GELU(h) D^-1| (h: the oracle's bf16 up output on the checked rows)."""

    def __init__(self, N, S, seed, g_or=None, use_dinv=True, clip=None):
        rng = np.random.default_rng([31, N, S, seed])
        self.gamma = rng.lognormal(0.0, 0.3, (T, S)).astype(np.float32)
        self.dinv = (np.float32(1.0) / rng.lognormal(0.0, 0.5, N).astype(np.float32)).astype(np.float32) \
            if use_dinv else None
        if clip is None:
            xt = O.bf16_bits_to_f32(g_or).astype(np.float64)
            if self.dinv is not None:
                xt = xt * self.dinv[None, :]
            clip = np.quantile(np.abs(xt), 0.999) * rng.lognormal(0.0, 0.2, T)
        self.clip = np.asarray(clip, dtype=np.float32)

    def device(self, t2s_dev, step):
        return B.ActParams(tok2stream=t2s_dev, gamma=f32_to_dev(self.gamma), step=step, act_bits=8,
                           range_mode=B.SQ_RANGE_STATIC, clip=f32_to_dev(self.clip),
                           dinv=f32_to_dev(self.dinv) if self.dinv is not None else None)


def run_fused(x, act, W, act_next, M, N):
    ws = B.alloc_workspace(B.SQ_VARIANT_FUSED, M, W.K, N, 8)
    qn = torch.full((M, N), 99, dtype=torch.int8, device="cuda")
    rn = torch.full((M,), float("nan"), dtype=torch.float32, device="cuda")
    B.sq_linear_w4a8_gelu_quant(x, act, W, act_next, qn, rn, ws)
    return qn, rn


def run_unfused(x, act, W, act_next, M, N):
    """The same chain from the separate entry points: the fused linear into
    bf16, GELU, the down projection's first kernel."""
    ws = B.alloc_workspace(B.SQ_VARIANT_FUSED, M, W.K, N, 8)
    h = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
    B.sq_linear_w4a8(x, act, W, h, B.SQ_OUT_BF16, ws)
    g = torch.empty_like(h)
    B.sq_gelu_bf16(h, g)
    qx, sc = B.act_buffers(M, N, 8)
    B.sq_quantize_act(g, act_next, qx, sc)
    return h, qx, sc


def check_chain(qn, rn, h_dev, qx_u, r_u, rows, h_or, qa):
    # fused == unfused GPU chain, every element
    assert torch.equal(qn, qx_u.view(torch.int8)), "fused codes differ from the unfused chain"
    assert torch.equal(rn.view(torch.int32), r_u.view(torch.int32)), "fused r differs from the unfused chain"
    ri = torch.as_tensor(rows, device=qn.device)
    # r against the oracle, bit for bit
    assert np.array_equal(rn[ri].cpu().numpy().view(np.uint32), qa["scale"].view(np.uint32))
    # codes against the oracle: equal wherever the bf16 up output agrees
    got = qn[ri].cpu().numpy().astype(np.int64)
    want = qa["codes"].astype(np.int64)
    hg = bits16(h_dev[ri])
    same_h = hg == h_or
    assert np.array_equal(got[same_h], want[same_h]), "codes differ where the bf16 up output agrees"
    d = np.abs(got - want)[~same_h]
    assert d.max(initial=0) <= 2
    assert (~same_h).mean() < 0.01, f"bf16 up output differs from the oracle's on {(~same_h).mean():.4f}"
    return int((~same_h).sum())


CHAIN = [  # name, M, K, N, stream counts
    ("300x2048x1024 all tiles split along K", 300, 2048, 1024, None),
    ("257x384x512 three stages never split", 257, 384, 512, None),
    ("2B up 4192x2048x8192", None, 2048, 8192, synth.TOKENS_2B),
    ("14B up 8384x5120x13824", None, 5120, 13824, synth.TOKENS_14B),
]


@pytest.mark.parametrize("name,M,K,N,counts", CHAIN, ids=[c[0] for c in CHAIN])
def test_gelu_quant_chain(name, M, K, N, counts):
    if counts is None:
        a = M // 6
        p = M // 10
        counts = (M - a - p, p, a)
    chain_case(counts, K, N, 128)


# At most 128 tokens the chain's up projection runs the weight-streaming GEMM
# with the GELU epilogue: 64 x 32 blocks, 64-channel strips, 32-row blocks
# with K split across workgroups (the epilogue then runs in the second
# kernel), and one weight step per channel (int32 sums, also through a split).
FEW = [  # name, stream counts, K, N, weight group
    ("2B up 64 action tokens", (0, 0, 64), 2048, 8192, 128),
    ("2B up 128 tokens 64-channel strips", (0, 64, 64), 2048, 8192, 128),
    ("64x8192x2048 32-row blocks split along K", (0, 0, 64), 8192, 2048, 128),
    ("100x2048x1024 one step per channel", (0, 36, 64), 2048, 1024, 2048),
    ("64x8192x512 one step per channel split along K", (0, 0, 64), 8192, 512, 8192),
    ("14B up 64 action tokens", (0, 0, 64), 5120, 13824, 128),
]


@pytest.mark.parametrize("name,counts,K,N,G", FEW, ids=[c[0] for c in FEW])
def test_gelu_quant_chain_few_tokens(name, counts, K, N, G):
    chain_case(counts, K, N, G)


# One weight step per output channel (the paper's weight format) on the tiled
# kernel: int32 sums over each tile's K range, converted once; with few tiles
# the ranges split and the second kernel applies the epilogue.
PC_CHAIN = [  # name, stream counts, K, N
    ("300x2048x1024 per channel, tiles split along K", (200, 40, 60), 2048, 1024),
    ("2B up 4192x2048x8192 per channel", synth.TOKENS_2B, 2048, 8192),
]


@pytest.mark.parametrize("name,counts,K,N", PC_CHAIN, ids=[c[0] for c in PC_CHAIN])
def test_gelu_quant_chain_per_channel(name, counts, K, N):
    chain_case(counts, K, N, K)


def chain_case(counts, K, N, G):
    L = synth.make_layer(K=K, N=N, stream_counts=counts, T=T, seed=[32, K, N], permute=True)
    M = L.M
    pw, W = oracle_weight(L, G)
    rows = tile_rows(M, seed=[33, M]) if M > 600 else np.arange(M)
    x = u16_to_dev(L.x_bits, torch.bfloat16)
    t2s_dev = i32_to_dev(L.tok2stream)
    step = 4
    for up_mode in (B.SQ_RANGE_DYNAMIC, B.SQ_RANGE_STATIC):
        act = act_params(L, step, 8, up_mode)
        res = O.linear(L.x_bits[rows], L.tok2stream[rows], L.gamma, step, pw["codes"], pw["w_scale"], G,
                       dinv=L.dinv, clip=L.clip, bias_bits=L.bias_bits, range_mode=up_mode, act_bits=8)
        h_or = O.f32_to_bf16_bits(res["y"])
        g_or = O.gelu_bf16(h_or)
        for use_dinv in (True, False):
            dp = DownParams(N, L.S, seed=[K, N, up_mode, use_dinv], g_or=g_or, use_dinv=use_dinv)
            act_next = dp.device(t2s_dev, step)
            h2, g2, qa = O.mlp_chain_codes(res["y"], L.tok2stream[rows], dp.gamma, step, dp.dinv, dp.clip)
            assert np.array_equal(h2, h_or) and np.array_equal(g2, g_or)
            codes = qa["codes"]
            assert np.abs(codes.astype(np.int64)).max() > 60, "threshold leaves the code range unused"
            qn, rn = run_fused(x, act, W, act_next, M, N)
            h_dev, qx_u, r_u = run_unfused(x, act, W, act_next, M, N)
            check_chain(qn, rn, h_dev, qx_u, r_u, rows, h_or, qa)
            del qn, rn, h_dev, qx_u, r_u


EXACT = [(300, 2048, 1024), (4192, 2048, 8192), (1000, 384, 640), (64, 2048, 8192), (64, 8192, 2048)]


@pytest.mark.parametrize("M,K,N", EXACT)
def test_gelu_quant_chain_exact(M, K, N):
    """Integer activations and power-of-two steps small enough that the up
    projection's outputs land mostly in GELU's curved range (|y| of a few
    units): the fp32 output is exact on both sides, so the chain's codes
    must equal the oracle's bit for bit on every checked row."""
    E = ExactLayer(M, K, N, 128, 8, seed=[41], w_exp=(-13, -10))
    x, act, W = E.device()
    rows = tile_rows(M, seed=[42, M])
    res = E.oracle(rows)
    y = res["y"]
    assert np.abs(y).max() < 1e4 and np.mean(np.abs(y) < 4) > 0.2, "outputs miss GELU's curved range"
    dp = DownParams(N, 3, seed=[43, M], clip=np.linspace(2.0, 9.0, T))
    act_next = dp.device(act.tok2stream, E.step)
    _, _, qa = O.mlp_chain_codes(y, E.t2s[rows], dp.gamma, E.step, dp.dinv, dp.clip)
    qn, rn = run_fused(x, act, W, act_next, M, N)
    ri = torch.as_tensor(rows, device="cuda")
    assert np.array_equal(qn[ri].cpu().numpy(), qa["codes"])
    assert np.array_equal(rn[ri].cpu().numpy().view(np.uint32), qa["scale"].view(np.uint32))
    # and the unfused chain agrees everywhere
    _, qx_u, r_u = run_unfused(x, act, W, act_next, M, N)
    assert torch.equal(qn, qx_u.view(torch.int8))
    assert torch.equal(rn.view(torch.int32), r_u.view(torch.int32))


# ---------------------------------------------------------------- 4-bit activations (the W4A4 chain)
def run_fused4(x, act, W, act_next, M, N):
    """The W4A4 up projection with the GELU epilogue.  At most 128 tokens the
    down projection's codes come packed with fp16 steps; above, as fp8 code
    bytes with fp32 steps and kc."""
    ws = B.alloc_workspace(B.SQ_VARIANT_FUSED, M, W.K, N, 4)
    if M <= 128:
        qn = torch.full((M, N // 2), 0x99, dtype=torch.uint8, device="cuda")
        sn = torch.full((M, N // 64), float("nan"), dtype=torch.float16, device="cuda")
        kn = None
    else:
        qn = torch.full((M, N), 0x55, dtype=torch.uint8, device="cuda")
        sn = torch.full((M, N // 64), float("nan"), dtype=torch.float32, device="cuda")
        kn = torch.full((M, N // 64), float("nan"), dtype=torch.float32, device="cuda")
    B.sq_linear_w4a4_gelu_quant(x, act, W, act_next, qn, sn, kn, ws)
    return qn, sn, kn


def run_unfused4(x, act, W, act_next, M, N):
    """sq_linear_w4a4 into bf16, sq_gelu_bf16, the down projection's first
    kernel (packed 4-bit codes, fp16 steps)."""
    ws = B.alloc_workspace(B.SQ_VARIANT_FUSED, M, W.K, N, 4)
    h = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
    B.sq_linear_w4a4(x, act, W, h, B.SQ_OUT_BF16, ws)
    g = torch.empty_like(h)
    B.sq_gelu_bf16(h, g)
    qx, sc = B.act_buffers(M, N, 4)
    B.sq_quantize_act(g, act_next, qx, sc)
    return h, qx, sc


def fp8_codes(b):
    """Codes from fp8 code bytes (sign and magnitude)."""
    b = b.astype(np.int64)
    return np.where(b & 0x80, -(b & 0x7F), b & 0x7F)


def check_chain4(qn, sn, kn, qx_u, sc_u, M, N):
    """The fused 4-bit chain against the unfused GPU chain, every element:
    packed form bit for bit; fp8 form the same codes, the fp16 steps widened,
    kc = -8 S sigma 2^-18 from the codes.  Returns the codes [M, N]."""
    codes_u = O.unpack_int4(qx_u.cpu().numpy())
    if M <= 128:
        assert torch.equal(qn, qx_u), "fused packed codes differ from the unfused chain"
        assert torch.equal(sn.view(torch.int16), sc_u.view(torch.int16)), "fused steps differ"
        return codes_u.astype(np.int64)
    codes = fp8_codes(qn.cpu().numpy())
    assert np.array_equal(codes, codes_u.astype(np.int64)), "fused fp8 codes differ from the unfused chain"
    sig_bits = bits16(sc_u)
    assert np.array_equal(sn.cpu().numpy(), sig_bits.view(np.float16).astype(np.float32)), "fused steps differ"
    assert np.array_equal(kn.cpu().numpy(), expected_kc(codes, sig_bits)), "kc differs"
    return codes


def chain_case4(counts, K, N, G):
    L = synth.make_layer(K=K, N=N, stream_counts=counts, T=T, seed=[34, K, N], permute=True)
    M = L.M
    pw, W = oracle_weight(L, G)
    rows = tile_rows(M, seed=[35, M]) if M > 600 else np.arange(M)
    x = u16_to_dev(L.x_bits, torch.bfloat16)
    t2s_dev = i32_to_dev(L.tok2stream)
    step = 6
    for up_mode in (B.SQ_RANGE_DYNAMIC, B.SQ_RANGE_STATIC):
        act = act_params(L, step, 4, up_mode)
        res = O.linear(L.x_bits[rows], L.tok2stream[rows], L.gamma, step, pw["codes"], pw["w_scale"], G,
                       dinv=L.dinv, clip=L.clip, bias_bits=L.bias_bits, range_mode=up_mode, act_bits=4)
        h_or = O.f32_to_bf16_bits(res["y"])
        g_or = O.gelu_bf16(h_or)
        for use_dinv in (True, False):
            dp = DownParams(N, L.S, seed=[K, N, up_mode, use_dinv, 4], g_or=g_or, use_dinv=use_dinv)
            act_next = B.ActParams(tok2stream=t2s_dev, gamma=f32_to_dev(dp.gamma), step=step, act_bits=4,
                                   range_mode=B.SQ_RANGE_STATIC, clip=f32_to_dev(dp.clip),
                                   dinv=f32_to_dev(dp.dinv) if dp.dinv is not None else None)
            _, _, qa = O.mlp_chain_codes(res["y"], L.tok2stream[rows], dp.gamma, step, dp.dinv, dp.clip, act_bits=4)
            assert np.abs(qa["codes"].astype(np.int64)).max() >= 6, "threshold leaves the code range unused"
            qn, sn, kn = run_fused4(x, act, W, act_next, M, N)
            h_dev, qx_u, sc_u = run_unfused4(x, act, W, act_next, M, N)
            codes = check_chain4(qn, sn, kn, qx_u, sc_u, M, N)
            # against the oracle: steps exact; codes equal wherever the bf16 up
            # output agrees, elsewhere within one code step
            assert np.array_equal(bits16(sc_u)[rows], qa["scale"])
            got = codes[rows]
            want = qa["codes"].astype(np.int64)
            same_h = bits16(h_dev)[rows] == h_or
            assert np.array_equal(got[same_h], want[same_h]), "codes differ where the bf16 up output agrees"
            assert np.abs(got - want)[~same_h].max(initial=0) <= 1
            assert (~same_h).mean() < 0.01
            del qn, sn, kn, h_dev, qx_u, sc_u


CHAIN4 = [  # name, stream counts, K, N
    ("64 action tokens 2048x8192 packed codes", (0, 0, 64), 2048, 8192),
    ("128 tokens 2048x8192 packed codes", (0, 64, 64), 2048, 8192),
    ("64 tokens 8192x2048 split along K, packed codes", (0, 0, 64), 8192, 2048),
    ("300x2048x1024 fp8 codes, tiles split along K", (200, 40, 60), 2048, 1024),
    ("2B up 4192x2048x8192 fp8 codes", synth.TOKENS_2B, 2048, 8192),
]


@pytest.mark.parametrize("name,counts,K,N", CHAIN4, ids=[c[0] for c in CHAIN4])
def test_gelu_quant_chain_4bit(name, counts, K, N):
    chain_case4(counts, K, N, 128)


@pytest.mark.parametrize("M,K,N", [(300, 2048, 1024), (64, 2048, 8192), (1000, 384, 640)])
def test_gelu_quant_chain_4bit_exact(M, K, N):
    """Integer 4-bit activations and power-of-two steps: the up projection's
    fp32 output is exact on both sides, so the chain's codes and steps equal
    the oracle's on every checked row (packed form at 64 tokens, fp8 form
    above 128)."""
    E = ExactLayer(M, K, N, 128, 4, seed=[44], w_exp=(-9, -6))
    x, act, W = E.device()
    rows = tile_rows(M, seed=[45, M])
    y = E.oracle(rows)["y"]
    assert np.mean(np.abs(y) < 4) > 0.2, "outputs miss GELU's curved range"
    dp = DownParams(N, 3, seed=[46, M], clip=np.linspace(2.0, 9.0, T))
    act_next = B.ActParams(tok2stream=act.tok2stream, gamma=f32_to_dev(dp.gamma), step=E.step, act_bits=4,
                           range_mode=B.SQ_RANGE_STATIC, clip=f32_to_dev(dp.clip), dinv=f32_to_dev(dp.dinv))
    _, _, qa = O.mlp_chain_codes(y, E.t2s[rows], dp.gamma, E.step, dp.dinv, dp.clip, act_bits=4)
    qn, sn, kn = run_fused4(x, act, W, act_next, M, N)
    _, qx_u, sc_u = run_unfused4(x, act, W, act_next, M, N)
    codes = check_chain4(qn, sn, kn, qx_u, sc_u, M, N)
    assert np.array_equal(codes[rows], qa["codes"].astype(np.int64))
    assert np.array_equal(bits16(sc_u)[rows], qa["scale"])


@pytest.mark.parametrize("M,K,N", [(300, 1024, 512), (4192, 8192, 2048)])
def test_gemm_w4a4_fp8_equals_packed(M, K, N):
    """The down projection's GEMM on the chain's fp8 form (sq_gemm_w4a4_fp8)
    equals sq_gemm_w4a4 on the same codes in the packed form, bit for bit
    (fp32 and bf16 outputs), with K split over idle workgroups where the
    tiles leave them (a workspace) and without."""
    rng = np.random.default_rng([47, M, K, N])
    counts = (M - M // 5, M // 10, M - (M - M // 5) - M // 10)
    L = synth.make_layer(K=K, N=N, stream_counts=counts, T=T, seed=[48, M], permute=True)
    _, W = oracle_weight(L, 128)
    codes = rng.integers(-7, 8, (M, K)).astype(np.int8)
    sig_bits = O.f32_to_f16_bits(rng.lognormal(-3.0, 0.5, (M, K // 64)).astype(np.float32))
    act = act_params(L, 2, 4, B.SQ_RANGE_DYNAMIC)
    packed = torch.from_numpy(O.pack_int4(codes)).cuda()
    sig16 = torch.from_numpy(sig_bits.view(np.int16)).view(torch.float16).cuda()
    f8 = np.where(codes < 0, 0x80 | (-codes.astype(np.int16)), codes.astype(np.int16)).astype(np.uint8)
    qf8 = torch.from_numpy(f8).cuda()
    sig32 = torch.from_numpy(sig_bits.view(np.float16).astype(np.float32)).cuda()
    kc = torch.from_numpy(expected_kc(codes.astype(np.int64), sig_bits)).cuda()
    for out, dt in ((B.SQ_OUT_F32, torch.float32), (B.SQ_OUT_BF16, torch.bfloat16)):
        for with_ws in (False, True):
            ws = B.alloc_workspace(B.SQ_VARIANT_GEMM, M, K, N, 4) if with_ws else None
            y0 = torch.full((M, N), float("nan"), dtype=dt, device="cuda")
            y1 = torch.full((M, N), float("nan"), dtype=dt, device="cuda")
            B.sq_gemm_w4a4(packed, sig16, act, W, y0, out, workspace=ws)
            B.sq_gemm_w4a4_fp8(qf8, sig32, kc, act, W, y1, out, workspace=ws)
            assert torch.equal(y0.view(torch.int16 if dt == torch.bfloat16 else torch.int32),
                               y1.view(torch.int16 if dt == torch.bfloat16 else torch.int32)), (out, with_ws)
