"""Parity at the C ABI's size limits: K = 32768 (the quantizer's longest rows,
the longest K loops), N = 2^20, and M = 2^24 rows, where row x channel offsets
pass 2^31 (every address computation must be 64-bit).  Full outputs where the
oracle is quick, sampled rows otherwise; codes bit-exact, fp32 outputs to the
summation-scale bound, bf16 to 1 ulp."""
import numpy as np
import pytest
import torch

from gpu_util import act_params, check_first_kernel_output, check_output, u16_to_dev, u8_to_dev
from oracle import sq_oracle as O
from paper_2609_39056_amd import binding as B
from paper_2609_39056_amd import synth

pytestmark = pytest.mark.gpu

F32, BF16 = B.SQ_OUT_F32, B.SQ_OUT_BF16
FUSED = {8: B.sq_linear_w4a8, 4: B.sq_linear_w4a4}


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.lib()


def split(M):
    a = max(M // 6, 0)
    p = max(M // 10, 0)
    return (M - a - p, p, a)


def dev_weight(w_nk, d, bias_bits, G=128):
    """Oracle-packed weights (w_nk: W^T, fp32 [N, K]) as device tensors."""
    pw = O.pack_weights(w_nk, d, G)
    W = B.Weight(qw=u8_to_dev(pw["qw"]), w_scale=u16_to_dev(pw["w_scale"].T, torch.float16), w_group=G,
                 bias=u16_to_dev(bias_bits, torch.bfloat16))
    return pw, W


def oracle_rows(xb, t2s, gamma, step, pw, dinv, clip, bias_bits, bits, G=128):
    return O.linear(xb, t2s, gamma, step, pw["codes"], pw["w_scale"], G, dinv=dinv, clip=clip,
                    bias_bits=bias_bits, range_mode=0, act_bits=bits)


def run_fused(bits, x, act, W, M, out):
    ws = B.alloc_workspace(B.SQ_VARIANT_FUSED, M, W.K, W.N, bits)
    y = torch.full((M, W.N), float("nan"), dtype=torch.float32 if out == F32 else torch.bfloat16, device="cuda")
    FUSED[bits](x, act, W, y, out, ws)
    torch.cuda.synchronize()
    return y, ws


@pytest.mark.parametrize("bits,G", [(8, 128), (4, 128), (8, 32768)])
@pytest.mark.parametrize("M", [37, 200])
def test_max_k(bits, G, M):
    """K = 32768: 37 tokens (weight-streaming kernel, K split across
    workgroups) and 200 (tiled kernel); with one weight step per channel the
    int32 sums span all 32768 channels.  Every output against the oracle."""
    K, N = 32768, 64
    L = synth.make_layer(K=K, N=N, stream_counts=split(M), T=3, seed=[20, M, K], permute=True)
    pw, W = dev_weight(L.w, L.d, L.bias_bits, G)
    act = act_params(L, 1, bits, 0)
    y, ws = run_fused(bits, u16_to_dev(L.x_bits, torch.bfloat16), act, W, M, F32)
    res = oracle_rows(L.x_bits, L.tok2stream, L.gamma, 1, pw, L.dinv, L.clip, L.bias_bits, bits, G)
    check_output(y, res, F32)
    check_first_kernel_output(ws, M, K, bits, G, res)


@pytest.mark.parametrize("bits,M", [(8, 3), (8, 200), (4, 200)])
def test_max_n(bits, M):
    """N = 2^20 output channels at K = 128: 32768 strips of the weight-streaming
    kernel (3 tokens), 16384 tiles of the tiled kernel (200 tokens, 8 rows
    checked; 4-bit codes on the fp8 matrix cores)."""
    K, N = 128, 1 << 20
    L = synth.make_layer(K=K, N=N, stream_counts=split(M), T=2, seed=[21, M], permute=True)
    pw, W = dev_weight(L.w, L.d, L.bias_bits)
    act = act_params(L, 0, bits, 0)
    y, _ = run_fused(bits, u16_to_dev(L.x_bits, torch.bfloat16), act, W, M, BF16)
    rows = np.arange(M) if M <= 8 else np.array([0, 1, 63, 64, 127, 128, 198, 199])
    res = oracle_rows(L.x_bits[rows], L.tok2stream[rows], L.gamma, 0, pw, L.dinv, L.clip, L.bias_bits, bits)
    check_output(y, res, BF16, rows=rows)


@pytest.mark.parametrize("bits", [8, 4])
def test_max_m(bits):
    """M = 2^24 tokens at K = 128 (X is 4 GiB; row * K reaches 2^31): the
    codes and outputs of 300 sampled rows, including the last ones."""
    M, K, N = 1 << 24, 128, 64
    a_n, p_n = 1 << 10, 1 << 9
    D = synth.device_layer(K, N, (M - a_n - p_n, p_n, a_n), T=3, seed=22)
    w_nk = D["w"].cpu().numpy()
    d = D["d"].cpu().numpy()
    bias_bits = D["bias"].view(torch.int16).cpu().numpy().view(np.uint16)
    pw, W = dev_weight(w_nk, d, bias_bits)
    act = B.ActParams(tok2stream=D["tok2stream"], gamma=D["gamma"], step=2, act_bits=bits, dinv=D["dinv"])
    y, ws = run_fused(bits, D["x"], act, W, M, BF16)
    rng = np.random.default_rng(0)
    rows = np.unique(np.concatenate([rng.integers(0, M, 280), [0, 1, (1 << 23) - 1, 1 << 23],
                                     np.arange(M - 16, M)])).astype(np.int64)
    ri = torch.as_tensor(rows, device="cuda")
    xb = D["x"][ri].view(torch.int16).cpu().numpy().view(np.uint16)
    t2s = D["tok2stream"][ri].cpu().numpy()
    gamma = D["gamma"].cpu().numpy()
    dinv = D["dinv"].cpu().numpy()
    res = oracle_rows(xb, t2s, gamma, 2, pw, dinv, None, bias_bits, bits)
    check_output(y, res, BF16, rows=rows)
    check_first_kernel_output(ws, M, K, bits, 128, res, rows=rows)
    del ws
    # the unfused path (one workgroup per row in its first kernel)
    wsu = B.alloc_workspace(B.SQ_VARIANT_UNFUSED, M, K, N, bits)
    y.fill_(float("nan"))
    B.sq_linear_unfused(D["x"], act, W, y, BF16, wsu)
    torch.cuda.synchronize()
    check_output(y, res, BF16, rows=rows)


def test_pack_weights_max():
    """The GPU weight packer at N = 2^20, K = 8192: 2^26 waves, 2^32
    work-items (32 GiB of fp32 weights, drawn on the device); 64 sampled
    output channels and the last one against the oracle's packing."""
    N, K, G = 1 << 20, 8192, 128
    gen = torch.Generator(device="cuda")
    gen.manual_seed(23)
    w = torch.randn((N, K), generator=gen, device="cuda") * 0.02
    d = torch.exp(torch.randn((K,), generator=gen, device="cuda") * 0.3)
    W = B.prepare_weight(w, d, G)
    torch.cuda.synchronize()
    cols = np.unique(np.concatenate([np.random.default_rng(1).integers(0, N, 64), [0, N - 1]])).astype(np.int64)
    ci = torch.as_tensor(cols, device="cuda")
    pw = O.pack_weights(w[ci].cpu().numpy(), d.cpu().numpy(), G)
    del w
    assert np.array_equal(W.qw.view(N, K // 2)[ci].cpu().numpy(), pw["qw"])
    steps = W.w_scale.view(K // G, N)[:, ci].t().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
    assert np.array_equal(steps, pw["w_scale"])
