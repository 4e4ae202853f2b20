"""Integer-exact checks of the int32 block accumulators of the production GEMM
kernels, through the same dispatch the fused linear and the benchmark use.

Sec. 4.4 accumulates C = Q_X Q_W in INT32 and dequantizes in the epilogue
(Eq. 10, generalised to K-blocks).  The fp32 bar of the other parity tests
(1e-5 of the summation scale) cannot see a +-1 error in one C^beta once the
blocks sum to more than about 1e5.  Here the inputs make every floating-point
step of the epilogue exact, so the output must EQUAL the exact value:

* activations are integers q scaled by powers of two: x = q / (gamma_s d_k^-1)
  with STATIC thresholds c = q_max, so Delta = 1, the quantizer returns q
  itself and r_i = 1 / gamma_s (8-bit) or sigma = 1, kappa = 1 / gamma_s
  (4-bit) are powers of two;
* every weight step Delta_W and (4-bit GEMM entry) activation step sigma is a
  power of two; no bias; fp32 output.

Then y_ij = r_i sum_beta C^beta_ij Delta_W[j, beta] (times sigma, kappa for
4-bit activations) is a sum of integers times powers of two.  When
sum_beta |C^beta| Delta_beta / min Delta < 2^24 (asserted on the data),
every partial sum of it is exactly representable in fp32, in any order, with
or without FMA, and across split-K partial sums: the GPU's fp32 output must be
bit-identical to the exact value, and so must the oracle's canonical fp32
epilogue.  A wrong C^beta anywhere moves y by at least the smallest step.

Cases cover every GEMM kernel the fused linear dispatches to: the tiled
16 x 16 kernel (8-bit, 128-wide groups), the tiled kernel with one step per
output channel (int32 sums over all of K, int32 split partials), the fp8
4-bit kernel, the int8-path 4-bit tiled kernel (the GEMM entry point), and the
weight-streaming kernel (8- and 4-bit, with and without its K split), at the
benchmark's full layer shapes (rows sampled for the oracle: every 128-row tile
is represented) and at 64 / 128 tokens.  The GEMM entry points additionally
take the full two's-complement code ranges (-128 and -8)."""
import numpy as np
import pytest
import torch

from gpu_util import check_first_kernel_output, f32_to_dev, i32_to_dev, u8_to_dev
from oracle import sq_oracle as O
from paper_2609_39056_amd import binding as B

pytestmark = pytest.mark.gpu

F32 = B.SQ_OUT_F32
T, S = 10, 3


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.lib()


def pow2_f16_bits(e):
    """fp16 bit patterns of 2^e (normal range)."""
    e = np.asarray(e, dtype=np.int64)
    assert np.all((e >= -14) & (e <= 15))
    return ((e + 15) << 10).astype(np.uint16)


def tile_rows(M, seed):
    """Rows checked against the oracle: the first, the last and two random
    rows of every 128-row tile, and every row of a ragged last tile."""
    if M <= 128:
        return np.arange(M)
    rng = np.random.default_rng(seed)
    rows = []
    for t0 in range(0, M, 128):
        t1 = min(M, t0 + 128)
        if t1 - t0 < 128:
            rows.extend(range(t0, t1))
        else:
            rows.extend([t0, t1 - 1, *rng.integers(t0, t1, 2)])
    return np.unique(np.asarray(rows, dtype=np.int64))


class ExactLayer:
    """Integer activations and power-of-two scales (see the module docstring)."""

    def __init__(self, M, K, N, G, bits, seed, w_lo=-7, w_exp=(-2, 2)):
        rng = np.random.default_rng([21, M, K, N, G, bits] + list(np.atleast_1d(seed)))
        qa = 127 if bits == 8 else 7
        self.M, self.K, self.N, self.G, self.bits = M, K, N, G, bits
        self.t2s = rng.integers(0, S, M).astype(np.int32)
        self.gamma = np.ldexp(np.float32(1.0), rng.integers(-1, 2, (T, S))).astype(np.float32)
        self.dinv = np.ldexp(np.float32(1.0), rng.integers(-2, 3, K)).astype(np.float32)
        self.clip = np.full(T, qa, dtype=np.float32)
        q = rng.integers(-qa, qa + 1, (M, K), dtype=np.int8)
        q[np.arange(M), rng.integers(0, K, M)] = np.where(rng.random(M) < 0.5, -qa, qa)  # both extremes occur
        self.q = q
        self.step = int(rng.integers(0, T))
        g = self.gamma[self.step, self.t2s]
        # x = q / (g dinv): exact in fp32 and in bf16 (|q| has at most 7 significant bits)
        x32 = q.astype(np.float32) * (np.float32(1.0) / g)[:, None] * (np.float32(1.0) / self.dinv)[None, :]
        u = x32.view(np.uint32)
        assert not np.any(u & 0xFFFF), "activation not exact in bf16"
        self.x_bits = (u >> 16).astype(np.uint16)
        self.cw = rng.integers(w_lo, 8, (N, K), dtype=np.int8)
        self.ws_bits = pow2_f16_bits(rng.integers(w_exp[0], w_exp[1], (N, K // G)))  # [N][K/G]

    def device(self, range_mode=B.SQ_RANGE_STATIC):
        act = B.ActParams(tok2stream=i32_to_dev(self.t2s), gamma=f32_to_dev(self.gamma), step=self.step,
                          act_bits=self.bits, range_mode=range_mode, clip=f32_to_dev(self.clip),
                          dinv=f32_to_dev(self.dinv))
        W = B.Weight(qw=u8_to_dev(O.pack_int4(self.cw)),
                     w_scale=torch.from_numpy(np.ascontiguousarray(self.ws_bits.T).view(np.int16))
                     .view(torch.float16).cuda(), w_group=self.G)
        x = torch.from_numpy(self.x_bits.view(np.int16)).view(torch.bfloat16).cuda()
        return x, act, W

    def oracle(self, rows):
        return O.linear(self.x_bits[rows], self.t2s[rows], self.gamma, self.step, self.cw, self.ws_bits, self.G,
                        dinv=self.dinv, clip=self.clip, range_mode=O.RANGE_STATIC, act_bits=self.bits)


def exact_value(C, scale_exp, w_exp, row_factor):
    """sum_beta C^beta * 2^(scale_exp + w_exp) * row_factor in fp64, exactly,
    and the check that fp32 represents every partial sum of it.
      C          int64 [nb, R, N] block sums
      scale_exp  int [R, nb] exponent of the activation step per block (0 for 8-bit)
      w_exp      int [N, nb] exponent of the weight step per block
      row_factor fp64 [R] power of two (r_i or kappa_i)."""
    emin = int(scale_exp.min()) + int(w_exp.min())
    units = np.zeros(C.shape[1:], dtype=np.int64)               # the sum in units of 2^emin
    mags = np.zeros(C.shape[1:], dtype=np.int64)
    for b in range(C.shape[0]):
        t = C[b] << (scale_exp[:, b][:, None] + w_exp[:, b][None, :] - emin)
        units += t
        mags += np.abs(t)
    assert mags.max() < 2**24, "inputs do not keep every partial sum exact in fp32"
    return np.ldexp(units.astype(np.float64), emin) * row_factor[:, None]


def w_exponents(ws_bits, nb, G, blk):
    """Exponent of each K-block's weight step, [N, nb]."""
    e = (ws_bits.astype(np.int64) >> 10) - 15
    return np.repeat(e, G // blk, axis=1)[:, :nb]


def check_exact(y_dev, rows, want):
    got = y_dev[torch.as_tensor(rows, device=y_dev.device)].cpu().numpy()
    assert np.all(np.isfinite(got))
    bad = got.astype(np.float64) != want
    assert not bad.any(), (f"{int(bad.sum())} outputs differ from the exact value; first at "
                           f"{np.argwhere(bad)[0]}: got {got[bad][0]!r}, want {want[bad][0]!r}")


# (name, bits, M, K, N, G): the tiled kernels at the benchmark's layer shapes
# (the 2B MLP at 4192 tokens, the 14B block at 8384), one weight step per
# output channel, and the weight-streaming kernel at 64 / 128 tokens (2B down
# splits K over 4 (8-bit) or 8 (4-bit) workgroups).
FUSED = [
    ("2B up A8 g128 (tiled 16x16, split tail)", 8, 4192, 2048, 8192, 128),
    ("2B down A8 g128", 8, 4192, 8192, 2048, 128),
    ("14B down A8 g128", 8, 8384, 13824, 5120, 128),
    ("14B qkv A8 g128", 8, 8384, 5120, 15360, 128),
    ("2B up A8 per-channel (int32 over K, split tail)", 8, 4192, 2048, 8192, 2048),
    ("2B down A8 per-channel", 8, 4192, 8192, 2048, 8192),
    ("14B down A8 per-channel", 8, 8384, 13824, 5120, 13824),
    ("2B up A4 (fp8 matrix cores)", 4, 4192, 2048, 8192, 128),
    ("2B down A4 (fp8)", 4, 4192, 8192, 2048, 128),
    ("14B down A4 (fp8)", 4, 8384, 13824, 5120, 128),
    ("14B out A4 per-channel (fp8)", 4, 8384, 5120, 5120, 5120),
    ("2B up A8 64 tokens (weight streaming)", 8, 64, 2048, 8192, 128),
    ("2B down A8 64 tokens (K split)", 8, 64, 8192, 2048, 128),
    ("2B qkv A8 128 tokens", 8, 128, 2048, 6144, 128),
    ("2B down A8 64 tokens per-channel (int32 split)", 8, 64, 8192, 2048, 8192),
    ("2B up A8 128 tokens per-channel", 8, 128, 2048, 8192, 2048),
    ("2B up A4 64 tokens", 4, 64, 2048, 8192, 128),
    ("2B down A4 64 tokens (K split)", 4, 64, 8192, 2048, 128),
    ("2B out A4 128 tokens", 4, 128, 2048, 2048, 128),
    ("14B down A4 97 tokens per-channel", 4, 97, 13824, 5120, 13824),
]


@pytest.mark.parametrize("name,bits,M,K,N,G", FUSED, ids=[f[0] for f in FUSED])
def test_fused_linear_exact(name, bits, M, K, N, G):
    """The fused linear (first kernel, then the GEMM the dispatch picks) on
    exact inputs: the output equals r_i sum_beta C^beta Delta_W (times kappa
    for 4-bit activations) exactly; the workspace codes equal q."""
    L = ExactLayer(M, K, N, G, bits, seed=0)
    x, act, W = L.device()
    ws = B.alloc_workspace(B.SQ_VARIANT_FUSED, M, K, N, bits)
    y = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
    (B.sq_linear_w4a8 if bits == 8 else B.sq_linear_w4a4)(x, act, W, y, F32, ws)
    torch.cuda.synchronize()
    rows = tile_rows(M, seed=M)
    res = L.oracle(rows)
    assert np.array_equal(res["codes"], L.q[rows]), "oracle codes differ from q (Delta = 1)"
    check_first_kernel_output(ws, M, K, bits, G, res, rows=rows)
    blk = res["G"]
    nb = K // blk
    g = L.gamma[L.step, L.t2s[rows]].astype(np.float64)
    want = exact_value(res["C"], np.zeros((len(rows), nb), np.int64), w_exponents(L.ws_bits, nb, G, blk), 1.0 / g)
    assert np.array_equal(res["y"].astype(np.float64), want), "oracle fp32 epilogue not exact"
    check_exact(y, rows, want)


# (bits, M, K, N, G, with_ws): the GEMM entry points on the full two's-
# complement code ranges; with a workspace the tiled kernels split leftover
# tiles along K and the weight-streaming kernel may split K.
GEMM = [
    (8, 4192, 2048, 8192, 128, True),
    (8, 4192, 2048, 8192, 128, False),
    (8, 1000, 8192, 2048, 8192, True),
    (8, 300, 13824, 512, 128, True),
    (8, 64, 8192, 2048, 128, True),
    (8, 100, 13824, 1024, 13824, True),
    (4, 4192, 2048, 2048, 128, True),
    (4, 600, 8192, 1024, 8192, True),
    (4, 64, 8192, 2048, 128, True),
    (4, 128, 5120, 5120, 5120, False),
]


@pytest.mark.parametrize("bits,M,K,N,G,with_ws", GEMM)
def test_gemm_entry_exact(bits, M, K, N, G, with_ws):
    """sq_gemm_w4a8 / sq_gemm_w4a4 on codes over the full int8 / int4 ranges
    (including -128 and -8), power-of-two row scales r (8-bit) or group steps
    sigma and gains (4-bit), power-of-two weight steps: outputs exact."""
    rng = np.random.default_rng([22, bits, M, K, N, G])
    L = ExactLayer(M, K, N, G, bits, seed=1, w_lo=-8)
    lo, hi = (-128, 128) if bits == 8 else (-8, 8)
    cx = rng.integers(lo, hi, (M, K), dtype=np.int8)
    _, act, W = L.device()
    rows = tile_rows(M, seed=M + 1)
    y = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
    ws = B.alloc_workspace(B.SQ_VARIANT_GEMM, M, K, N, bits) if with_ws else None
    if bits == 8:
        r_exp = rng.integers(-3, 2, M)
        r = np.ldexp(np.float32(1.0), r_exp).astype(np.float32)
        B.sq_gemm_w4a8(torch.from_numpy(cx).cuda(), f32_to_dev(r), W, y, F32, workspace=ws)
        blk = G
        sexp = np.zeros((len(rows), K // blk), np.int64)
        rowf = r[rows].astype(np.float64)
    else:
        s_exp = rng.integers(-1, 2, (M, K // 64))
        sigma = pow2_f16_bits(s_exp)
        B.sq_gemm_w4a4(u8_to_dev(O.pack_int4(cx)), torch.from_numpy(sigma.view(np.int16)).view(torch.float16).cuda(),
                       act, W, y, F32, workspace=ws)
        blk = 64
        sexp = s_exp[rows]
        rowf = 1.0 / L.gamma[L.step, L.t2s[rows]].astype(np.float64)
    torch.cuda.synchronize()
    C = O.block_acc(cx[rows], L.cw, blk)
    want = exact_value(C, sexp, w_exponents(L.ws_bits, K // blk, G, blk), rowf)
    # the oracle's canonical fp32 epilogue is exact on these inputs as well
    scale = r[rows] if bits == 8 else sigma[rows]
    y_or, _, _ = O.epilogue(C, bits, scale, (1.0 / L.gamma[L.step, L.t2s[rows]]).astype(np.float32), L.ws_bits, G)
    assert np.array_equal(y_or.astype(np.float64), want), "oracle fp32 epilogue not exact"
    check_exact(y, rows, want)
