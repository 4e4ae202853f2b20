"""The STATIC single-kernel W4A8 linear (sq_linear_w4a8_static1): the
weight-streaming GEMM quantizing X itself, stage by stage in LDS.

Its codes never reach memory, so parity is shown three ways: the outputs equal
those of the two-kernel linear with the same K-split plan (whose codes are
checked bit-exactly elsewhere) bit for bit; they lie within the oracle's bar; and on
exact-arithmetic inputs (integer activations, power-of-two scales) they equal
the exact value, which requires every code and int32 block sum to be right."""
import numpy as np
import pytest
import torch

from gpu_util import act_params, check_output, oracle_weight, u16_to_dev
from oracle import sq_oracle as O
from paper_2609_39056_amd import binding as B
from paper_2609_39056_amd import synth
from test_exact_accum_gpu import ExactLayer, check_exact, exact_value, tile_rows, w_exponents

pytestmark = pytest.mark.gpu

F32, BF16, F16 = B.SQ_OUT_F32, B.SQ_OUT_BF16, B.SQ_OUT_F16
TORCH_OUT = {F32: torch.float32, BF16: torch.bfloat16, F16: torch.float16}


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.lib()


def split(M):
    a = max(M // 6, 0)
    p = max(M // 10, 0)
    return (M - a - p, p, a)


@pytest.mark.parametrize("M,K,N,G", [(1, 256, 64, 128), (37, 2048, 512, 128), (64, 2048, 8192, 128),
                                     (65, 1024, 256, 1024), (100, 13824, 128, 128), (128, 8192, 2048, 8192),
                                     (64, 8192, 2048, 128), (128, 2048, 6144, 2048)])
@pytest.mark.parametrize("use_d", [True, False])
def test_static1_equals_two_kernel_linear(M, K, N, G, use_d):
    """Bit-identical to sq_linear_w4a8 in STATIC mode (same codes, same GEMM),
    with and without a workspace (K split), fp32 and bf16 outputs; and within
    the oracle's bar."""
    L = synth.make_layer(K=K, N=N, stream_counts=split(M), T=4, seed=[41, M, K, N, G], permute=True)
    pw, W = oracle_weight(L, G)
    step = 2
    act = act_params(L, step, 8, B.SQ_RANGE_STATIC, use_dinv=use_d)
    x = u16_to_dev(L.x_bits, torch.bfloat16)
    res = O.linear(L.x_bits, L.tok2stream, L.gamma, step, pw["codes"], pw["w_scale"], G,
                   dinv=L.dinv if use_d else None, clip=L.clip, bias_bits=L.bias_bits,
                   range_mode=O.RANGE_STATIC, act_bits=8)
    for out in (F32, BF16):
        view = torch.int32 if out == F32 else torch.int16
        for with_ws in (False, True):
            # the two kernels with the same K-split plan: the fused call with a
            # workspace, or the first kernel then the GEMM without one
            y2 = torch.full((M, N), float("nan"), dtype=TORCH_OUT[out], device="cuda")
            if with_ws:
                B.sq_linear_w4a8(x, act, W, y2, out, B.alloc_workspace(B.SQ_VARIANT_FUSED, M, K, N, 8))
            else:
                qx, sc = B.act_buffers(M, K, 8)
                B.sq_quantize_act(x, act, qx, sc)
                B.sq_gemm_w4a8(qx, sc, W, y2, out)
            wsg = B.alloc_workspace(B.SQ_VARIANT_GEMM, M, K, N, 8) if with_ws else None
            y1 = torch.full((M, N), float("nan"), dtype=TORCH_OUT[out], device="cuda")
            B.sq_linear_w4a8_static1(x, act, W, y1, out, wsg)
            torch.cuda.synchronize()
            assert torch.equal(y1.view(view), y2.view(view)), (out, with_ws)
            check_output(y1, res, out)


@pytest.mark.parametrize("M,K,N,G", [(64, 2048, 8192, 128), (64, 8192, 2048, 128), (128, 13824, 1024, 13824),
                                     (33, 5120, 512, 128)])
def test_static1_exact(M, K, N, G):
    """Integer activations and power-of-two scales: the output equals
    r_i sum_beta C^beta Delta_W exactly (every code, block sum and step right)."""
    L = ExactLayer(M, K, N, G, 8, seed=5)
    x, act, W = L.device()
    wsg = B.alloc_workspace(B.SQ_VARIANT_GEMM, M, K, N, 8)
    y = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
    B.sq_linear_w4a8_static1(x, act, W, y, F32, wsg)
    torch.cuda.synchronize()
    rows = tile_rows(M, seed=M)
    res = L.oracle(rows)
    g = L.gamma[L.step, L.t2s[rows]].astype(np.float64)
    want = exact_value(res["C"], np.zeros((len(rows), K // res["G"]), np.int64),
                       w_exponents(L.ws_bits, K // res["G"], G, res["G"]), 1.0 / g)
    check_exact(y, rows, want)


def test_static1_degenerate_rows():
    """All-zero rows, a threshold below every element (all codes saturate),
    bf16 subnormals and huge values, against the two-kernel linear."""
    K, N = 256, 128
    rows = [np.zeros(K), np.full(K, 2.0**-130) * np.sign(np.arange(K) - 100.5), np.linspace(-1e30, 1e30, K),
            np.random.default_rng(0).standard_normal(K) * 1e-3]
    xb = O.f32_to_bf16_bits(np.stack(rows).astype(np.float32))
    M = xb.shape[0]
    L = synth.make_layer(K=K, N=N, stream_counts=(2, 1, 1), T=2, seed=3)
    _, W = oracle_weight(L, 128)
    x = u16_to_dev(xb, torch.bfloat16)
    t2s = torch.tensor([0, 1, 2, 0], dtype=torch.int32, device="cuda")
    gamma = torch.tensor([[1.0, 0.5, 3.0], [1.25, 1.0, 0.75]], device="cuda")
    for clip in ([1e-6, 1e-6], [2.0, 2.0]):
        act = B.ActParams(tok2stream=t2s, gamma=gamma, step=1, act_bits=8, range_mode=B.SQ_RANGE_STATIC,
                          clip=torch.tensor(clip, device="cuda"), dinv=None)
        y1 = torch.full((M, N), float("nan"), device="cuda")
        y2 = torch.full((M, N), float("nan"), device="cuda")
        B.sq_linear_w4a8_static1(x, act, W, y1, F32)
        B.sq_linear_w4a8(x, act, W, y2, F32, B.alloc_workspace(B.SQ_VARIANT_FUSED, M, K, N, 8))
        torch.cuda.synchronize()
        assert torch.equal(y1.view(torch.int32), y2.view(torch.int32)), clip
