"""Parity of the HIP path (through the C ABI) with the CPU oracle.

Integers (codes, packed bytes, int32 block accumulators) and stored scales
must match bit-exactly; fp32 outputs within 1e-5 of the summation scale
(and 1e-5 relative where the sum does not cancel); bf16 / fp16 outputs within
1 ulp of the oracle's value cast the same way."""
import numpy as np
import pytest
import torch

from gpu_util import (act_params, bits16, check_first_kernel_output, check_output, f32_to_dev, i32_to_dev,
                      oracle_weight, u16_to_dev, u8_to_dev)
from oracle import sq_oracle as O
from paper_2609_39056_amd import binding as B
from paper_2609_39056_amd import synth

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


def layer(M, K, N, seed, T=3, permute=True, **kw):
    return synth.make_layer(K=K, N=N, stream_counts=split(M), T=T, seed=seed, permute=permute, **kw)


def xdev(L, rows=None):
    xb = L.x_bits if rows is None else L.x_bits[rows]
    return u16_to_dev(xb, torch.bfloat16)


# ------------------------------------------------------------------ first kernel
@pytest.mark.parametrize("bits,mode", [(8, 0), (8, 1), (4, 0), (4, 1)])
@pytest.mark.parametrize("K,M", [(128, 5), (256, 88), (2048, 67), (5120, 33), (8192, 40), (13824, 9)])
def test_quantize_bitexact(bits, mode, K, M):
    L = layer(M, K, 64, seed=[1, K, M])
    x = xdev(L)
    for step in (0, 2):
        for use_dinv in (True, False):
            act = act_params(L, step, bits, mode, use_dinv=use_dinv)
            qx, sc = B.act_buffers(M, K, bits)
            B.sq_quantize_act(x, act, qx, sc)
            ref = O.quantize_act(L.x_bits, L.tok2stream, L.gamma, step, dinv=L.dinv if use_dinv else None,
                                 clip=L.clip, range_mode=mode, act_bits=bits)
            assert np.array_equal(qx.cpu().numpy().view(np.uint8), ref["qx"].view(np.uint8))
            if bits == 8:
                assert np.array_equal(sc.cpu().numpy().view(np.uint32), ref["scale"].view(np.uint32))
            else:
                assert np.array_equal(bits16(sc), ref["scale"])


@pytest.mark.parametrize("bits", [8, 4])
@pytest.mark.parametrize("K,M", [(2560, 2051), (5120, 2049), (8192, 2050), (10240, 2051), (13824, 2048)])
def test_quantize_many_rows(bits, K, M):
    """Thousands of rows of the lengths the layers use, with a ragged row
    count (not a multiple of the rows per workgroup) and rows whose chunks
    leave lanes idle (2560 channels): codes and scales bit-exact, DYNAMIC and
    STATIC, with and without the channel scaling."""
    L = layer(M, K, 64, seed=[2, K, M])
    x = xdev(L)
    for mode in (0, 1):
        for use_dinv in (True, False):
            act = act_params(L, 1, bits, mode, use_dinv=use_dinv)
            qx, sc = B.act_buffers(M, K, bits)
            B.sq_quantize_act(x, act, qx, sc)
            ref = O.quantize_act(L.x_bits, L.tok2stream, L.gamma, 1, dinv=L.dinv if use_dinv else None,
                                 clip=L.clip, range_mode=mode, act_bits=bits)
            assert np.array_equal(qx.cpu().numpy().view(np.uint8), ref["qx"].view(np.uint8)), (mode, use_dinv)
            if bits == 8:
                assert np.array_equal(sc.cpu().numpy().view(np.uint32), ref["scale"].view(np.uint32))
            else:
                assert np.array_equal(bits16(sc), ref["scale"])


@pytest.mark.parametrize("bits", [8, 4])
def test_quantize_degenerate_rows(bits):
    """All-zero rows, a single non-zero element, bf16 subnormal magnitudes (the
    step underflows into fp32 subnormals and its reciprocal overflows), huge
    values, and STATIC thresholds below every element."""
    K = 256
    rows = []
    rows.append(np.zeros(K))
    r = np.zeros(K); r[17] = -3.5; rows.append(r)
    rows.append(np.full(K, 2.0**-130) * np.sign(np.arange(K) - 100.5))
    rows.append(np.linspace(-1e30, 1e30, K))
    rows.append(np.random.default_rng(0).standard_normal(K) * 1e-3)
    x = np.stack(rows).astype(np.float32)
    xb = O.f32_to_bf16_bits(x)
    M = xb.shape[0]
    t2s = np.array([0, 1, 2, 0, 1], np.int32)
    gamma = np.array([[1.0, 0.5, 3.0], [1.25, 1.0, 0.75]], np.float32)
    clip = np.array([1e-6, 2.0], np.float32)
    for mode in (0, 1):
        for step in (0, 1):
            act = B.ActParams(tok2stream=i32_to_dev(t2s), gamma=f32_to_dev(gamma), step=step, act_bits=bits,
                              range_mode=mode, clip=f32_to_dev(clip), dinv=None)
            qx, sc = B.act_buffers(M, K, bits)
            B.sq_quantize_act(u16_to_dev(xb, torch.bfloat16), act, qx, sc)
            ref = O.quantize_act(xb, t2s, gamma, step, clip=clip, range_mode=mode, act_bits=bits)
            assert np.array_equal(qx.cpu().numpy().view(np.uint8), ref["qx"].view(np.uint8)), (mode, step)
            if bits == 8:
                assert np.array_equal(sc.cpu().numpy().view(np.uint32), ref["scale"].view(np.uint32))
            else:
                assert np.array_equal(bits16(sc), ref["scale"])


# ------------------------------------------------------------------ weight preparation
@pytest.mark.parametrize("K,N,G", [(256, 256, 128), (256, 256, 256), (2048, 512, 128), (5120, 192, 128),
                                   (13824, 64, 13824), (384, 64, 384)])
def test_pack_weights_bitexact(K, N, G):
    L = layer(16, K, N, seed=[2, K, N])
    for use_d in (True, False):
        d = L.d if use_d else None
        ref = O.pack_weights(L.w, d, G)
        W = B.prepare_weight(f32_to_dev(L.w), f32_to_dev(L.d) if use_d else None, G)
        assert np.array_equal(W.qw.cpu().numpy(), ref["qw"])
        assert np.array_equal(bits16(W.w_scale), ref["w_scale"].T)  # group-major


# ------------------------------------------------------------------ int32 accumulators
@pytest.mark.parametrize("bits", [8, 4])
@pytest.mark.parametrize("M,K,N,G", [(88, 256, 256, 128), (1, 256, 64, 128), (63, 384, 192, 128),
                                     (130, 512, 320, 256), (200, 1024, 128, 1024), (257, 2048, 256, 128)])
def test_block_acc_bitexact(bits, M, K, N, G):
    """The fused main loop's int32 block accumulators, on random codes over the
    full two's-complement ranges (including -128 and -8)."""
    rng = np.random.default_rng([3, M, K, N, G, bits])
    if bits == 8:
        cx = rng.integers(-128, 128, size=(M, K)).astype(np.int8)
        qx = torch.from_numpy(cx).cuda()
    else:
        cx = rng.integers(-8, 8, size=(M, K)).astype(np.int8)
        qx = u8_to_dev(O.pack_int4(cx))
    cw = rng.integers(-8, 8, size=(N, K)).astype(np.int8)
    W = B.Weight(qw=u8_to_dev(O.pack_int4(cw)), w_scale=torch.ones((K // G, N), dtype=torch.float16, device="cuda"),
                 w_group=G)
    blk = G if bits == 8 else 64
    acc = torch.full((K // blk, M, N), 0x7EADBEEF, dtype=torch.int32, device="cuda")
    B.sq_debug_block_acc_i32(qx, bits, W, acc)
    ref = O.block_acc(cx, cw, blk)
    assert np.array_equal(acc.cpu().numpy().astype(np.int64), ref)


# ------------------------------------------------------------------ whole linear
def run_linear(fn, L, act, W, out, M=None, rows=None):
    M = L.M if M is None else M
    variant = B.SQ_VARIANT_UNFUSED if fn is B.sq_linear_unfused else B.SQ_VARIANT_FUSED
    ws = B.alloc_workspace(variant, M, W.K, W.N, act.act_bits)
    y = torch.full((M, W.N), float("nan"), dtype=TORCH_OUT[out], device="cuda")
    fn(xdev(L, rows), act, W, y, out, ws)
    return y, ws


def oracle_linear(L, step, bits, mode, pw, G, with_bias=True, rows=None):
    xb = L.x_bits if rows is None else L.x_bits[rows]
    t2s = L.tok2stream if rows is None else L.tok2stream[rows]
    return O.linear(xb, t2s, L.gamma, step, pw["codes"], pw["w_scale"], G, dinv=L.dinv, clip=L.clip,
                    bias_bits=L.bias_bits if with_bias else None, range_mode=mode, act_bits=bits)


FUSED = {8: B.sq_linear_w4a8, 4: B.sq_linear_w4a4}


@pytest.mark.parametrize("bits", [8, 4])
@pytest.mark.parametrize("mode", [0, 1])
@pytest.mark.parametrize("out", [F32, BF16, F16])
@pytest.mark.parametrize("G", [128, 256])
def test_linear_small_layer(bits, mode, out, G):
    """The 88-token 256 x 256 layer (64 video, 8 proprio, 16 action tokens,
    2 denoising steps), fused and unfused."""
    L = synth.make_layer(K=256, N=256, stream_counts=(64, 8, 16), T=2, seed=0)
    pw, W = oracle_weight(L, G)
    for step in (0, 1):
        act = act_params(L, step, bits, mode)
        res = oracle_linear(L, step, bits, mode, pw, G)
        for fn in (FUSED[bits], B.sq_linear_unfused):
            y, ws = run_linear(fn, L, act, W, out)
            check_output(y, res, out)
            if fn is not B.sq_linear_unfused:  # the first kernel's codes and scales, from the workspace
                check_first_kernel_output(ws, L.M, L.K, bits, G, res)


@pytest.mark.parametrize("bits", [8, 4])
@pytest.mark.parametrize("M,K,N,G,bias", [(1, 256, 64, 128, True), (63, 384, 192, 384, True),
                                          (130, 2048, 320, 128, False), (200, 1024, 128, 1024, True),
                                          (97, 13824, 64, 128, True), (70, 1664, 192, 128, True)])
def test_linear_shapes(bits, M, K, N, G, bias):
    """Ragged M and N tiles, a weight step per output channel (G = K, the
    paper's granularity), no bias, the largest K.  With fewer output tiles
    than workgroup slots the tiles are split along K: 1664 = 13 stages gives
    uneven ranges."""
    L = layer(M, K, N, seed=[4, M, K, N])
    pw, W = oracle_weight(L, G, with_bias=bias)
    act = act_params(L, 1, bits, 0)
    res = oracle_linear(L, 1, bits, 0, pw, G, with_bias=bias)
    for fn in (FUSED[bits], B.sq_linear_unfused):
        y, _ = run_linear(fn, L, act, W, F32)
        check_output(y, res, F32)


@pytest.mark.parametrize("bits", [8, 4])
@pytest.mark.parametrize("with_ws", [False, True])
def test_gemm_entry_points(bits, with_ws):
    """The second kernel alone, fed the oracle's codes and scales; without a
    workspace every tile is computed whole, with one the tiles are split along
    K (partial sums added by the second kernel)."""
    L = layer(150, 1024, 192, seed=5)
    pw, W = oracle_weight(L, 128)
    res = oracle_linear(L, 2, bits, 0, pw, 128)
    y = torch.empty((L.M, L.N), dtype=torch.float32, device="cuda")
    ws = B.alloc_workspace(B.SQ_VARIANT_GEMM, L.M, L.K, L.N, bits) if with_ws else None
    if bits == 8:
        B.sq_gemm_w4a8(torch.from_numpy(res["qx"]).cuda(), f32_to_dev(res["scale"]), W, y, F32, workspace=ws)
    else:
        B.sq_gemm_w4a4(u8_to_dev(res["qx"]), u16_to_dev(res["scale"], torch.float16), act_params(L, 2, 4, 0), W,
                       y, F32, workspace=ws)
    check_output(y, res, F32)


@pytest.mark.parametrize("bits", [8, 4])
@pytest.mark.parametrize("M,K,N", [(1, 2048, 2048), (2, 128, 64), (33, 8192, 2048), (64, 2048, 6144),
                                   (65, 5120, 320), (128, 1024, 1024), (100, 13824, 128), (128, 512, 8192),
                                   (100, 1024, 8448)])
@pytest.mark.parametrize("out", [F32, BF16])
@pytest.mark.parametrize("per_channel", [False, True])
def test_few_tokens(bits, M, K, N, out, per_channel):
    """Layers of at most 128 tokens (the action and proprio streams alone)
    take the weight-streaming kernel, with 128-wide weight groups or one step
    per output channel (8-bit: int32 sums over all of K, exact across the
    waves and split ranges).  Fused linear, and the second kernel alone
    without a workspace (K never split) and with one (K split across
    workgroups when that is faster: 8192 and 13824 channels here).  Blocks of
    32 rows (few output channels), 64 x 32, and 64 x 64 where 64 x 32 blocks
    would not all run at once (8192 channels at 128 tokens with 8-bit codes,
    8448 at 100 tokens with both widths)."""
    L = layer(M, K, N, seed=[9, M, K, N])
    G = K if per_channel else 128
    pw, W = oracle_weight(L, G)
    act = act_params(L, 1, bits, 0)
    res = oracle_linear(L, 1, bits, 0, pw, G)
    y, _ = run_linear(FUSED[bits], L, act, W, out)
    check_output(y, res, out)
    for with_ws in (False, True):
        ws = B.alloc_workspace(B.SQ_VARIANT_GEMM, L.M, L.K, L.N, bits) if with_ws else None
        y = torch.full((L.M, L.N), float("nan"), dtype=TORCH_OUT[out], device="cuda")
        if bits == 8:
            B.sq_gemm_w4a8(torch.from_numpy(res["qx"]).cuda(), f32_to_dev(res["scale"]), W, y, out, workspace=ws)
        else:
            B.sq_gemm_w4a4(u8_to_dev(res["qx"]), u16_to_dev(res["scale"], torch.float16), act, W, y, out,
                           workspace=ws)
        check_output(y, res, out)


@pytest.mark.parametrize("M,K,N", [(4192, 1024, 2048), (300, 2048, 384), (1000, 8192, 256), (64, 2048, 512),
                                   (129, 256, 128), (200, 512, 64)])
@pytest.mark.parametrize("out", [F32, BF16])
def test_per_channel_weights(M, K, N, out):
    """One weight step per output channel (G = K, the paper's weight format)
    with 8-bit activations: int32 sums over all of K in the pipelined kernel.
    4192 x 2048 outputs are 528 tiles, 512 computed whole and 16 split along
    K (int32 partial sums added by the second kernel); the smaller layers are
    split entirely, 256 channels (two stages) not at all.  Fused linear, and
    the second kernel alone without and with a workspace."""
    L = layer(M, K, N, seed=[13, M, K, N])
    pw, W = oracle_weight(L, K)
    act = act_params(L, 1, 8, 0)
    res = oracle_linear(L, 1, 8, 0, pw, K)
    y, _ = run_linear(B.sq_linear_w4a8, L, act, W, out)
    check_output(y, res, out)
    for with_ws in (False, True):
        ws = B.alloc_workspace(B.SQ_VARIANT_GEMM, L.M, L.K, L.N, 8) if with_ws else None
        y = torch.full((L.M, L.N), float("nan"), dtype=TORCH_OUT[out], device="cuda")
        B.sq_gemm_w4a8(torch.from_numpy(res["qx"]).cuda(), f32_to_dev(res["scale"]), W, y, out, workspace=ws)
        check_output(y, res, out)


@pytest.mark.parametrize("M,K,N,G", [(4192, 1024, 2048, 128), (300, 2048, 384, 128), (200, 1024, 128, 1024),
                                     (129, 256, 192, 128), (1000, 8192, 256, 8192)])
def test_a4_fp8_path_equals_int8_path(M, K, N, G):
    """4-bit activations on the fp8 matrix cores (the fused linear with more
    than 128 tokens or wide weight groups) against the int8 path (the first
    kernel's packed codes, then sq_gemm_w4a4): the first kernel's codes,
    steps and kc against the oracle, and the outputs bit for bit equal,
    with whole tiles, split tails, ragged M and N, and per-channel steps."""
    L = layer(M, K, N, seed=[14, M, K, N], outlier_frac=(0.01, 0.02, 0.05))
    pw, W = oracle_weight(L, G)
    act = act_params(L, 2, 4, 0)
    y, ws = run_linear(B.sq_linear_w4a4, L, act, W, F32)
    rows = synth.stratified_rows(L.tok2stream, 64, seed=1) if M > 1000 else None
    res = oracle_linear(L, 2, 4, 0, pw, G, rows=rows)
    check_first_kernel_output(ws, M, K, 4, G, res, rows=rows)
    check_output(y, res, F32, rows=rows)
    qx, sc = B.act_buffers(M, K, 4)
    B.sq_quantize_act(xdev(L), act, qx, sc)
    y_int = torch.full_like(y, float("nan"))
    B.sq_gemm_w4a4(qx, sc, act, W, y_int, F32, workspace=B.alloc_workspace(B.SQ_VARIANT_GEMM, M, K, N, 4))
    torch.cuda.synchronize()
    assert torch.equal(y.view(torch.int32), y_int.view(torch.int32))


@pytest.mark.parametrize("bits", [8, 4])
def test_gpu_prepared_weights_chain(bits):
    """Weights folded and packed on the GPU (sq_pack_weights), then the fused
    linear: equals the oracle's chain from the fp32 weight."""
    L = layer(100, 1024, 256, seed=6)
    W = B.prepare_weight(f32_to_dev(L.w), f32_to_dev(L.d), 128, bias=u16_to_dev(L.bias_bits, torch.bfloat16))
    pw = O.pack_weights(L.w, L.d, 128)
    act = act_params(L, 0, bits, 0)
    y, _ = run_linear(FUSED[bits], L, act, W, BF16)
    check_output(y, oracle_linear(L, 0, bits, 0, pw, 128), BF16)


@pytest.mark.parametrize("bits", [8, 4])
def test_deterministic(bits):
    L = layer(300, 2048, 512, seed=7)
    _, W = oracle_weight(L, 128)
    act = act_params(L, 1, bits, 0)
    y1, _ = run_linear(FUSED[bits], L, act, W, F32)
    y2, _ = run_linear(FUSED[bits], L, act, W, F32)
    assert torch.equal(y1.view(torch.int32), y2.view(torch.int32))


# ------------------------------------------------------------------ full-size layers, sampled rows
# (name, bit widths, tokens per sample, batch, K, N, outlier fraction(s)):
# every linear of the 2B (4192 tokens) and 14B (8384 tokens) configurations,
# the 4-bit 2B linears with per-stream outliers of 1 / 2 / 5 %, the batch-4
# sweep's row count (16768 tokens), and one GPU's column shard of the 14B up
# projection at 8-way tensor parallelism.
FULL = [
    ("2B up", (8, 4), synth.TOKENS_2B, 1, 2048, 8192, 0.02),
    ("2B down", (8,), synth.TOKENS_2B, 1, 8192, 2048, 0.02),
    ("2B qkv outliers 1/2/5%", (4,), synth.TOKENS_2B, 1, 2048, 6144, (0.01, 0.02, 0.05)),
    ("2B out outliers 1/2/5%", (4,), synth.TOKENS_2B, 1, 2048, 2048, (0.01, 0.02, 0.05)),
    ("2B up outliers 1/2/5%", (4,), synth.TOKENS_2B, 1, 2048, 8192, (0.01, 0.02, 0.05)),
    ("2B down outliers 1/2/5%", (4,), synth.TOKENS_2B, 1, 8192, 2048, (0.01, 0.02, 0.05)),
    ("2B up batch 4", (8, 4), synth.TOKENS_2B, 4, 2048, 8192, 0.02),
    ("14B qkv", (8, 4), synth.TOKENS_14B, 1, 5120, 15360, 0.02),
    ("14B out", (8, 4), synth.TOKENS_14B, 1, 5120, 5120, 0.02),
    ("14B up", (8, 4), synth.TOKENS_14B, 1, 5120, 13824, 0.02),
    ("14B down", (8, 4), synth.TOKENS_14B, 1, 13824, 5120, 0.02),
    ("14B up TP8 shard", (8, 4), synth.TOKENS_14B, 1, 5120, 1728, 0.02),
]


@pytest.mark.parametrize("name,bits_list,tokens,batch,K,N,outl", FULL, ids=[f[0] for f in FULL])
def test_full_size_sampled_rows(name, bits_list, tokens, batch, K, N, outl):
    """Full-size layers in the launch configuration the benchmark times, with
    fp32 and bf16 outputs; the oracle checks every proprio / action row and
    256 random video rows, and the first kernel's codes and scales of those
    rows are read back from the workspace."""
    L = synth.make_layer(K=K, N=N, stream_counts=tokens, T=10, seed=[8, K, N, batch], outlier_frac=outl,
                         batch=batch)
    pw, W = oracle_weight(L, 128)
    step = 7
    rows = synth.stratified_rows(L.tok2stream, 256, seed=0)
    x = xdev(L)
    for bits in bits_list:
        act = act_params(L, step, bits, 0)
        res = oracle_linear(L, step, bits, 0, pw, 128, rows=rows)
        ws = B.alloc_workspace(B.SQ_VARIANT_FUSED, L.M, K, N, bits)
        for out in (F32, BF16):
            y = torch.full((L.M, N), float("nan"), dtype=TORCH_OUT[out], device="cuda")
            FUSED[bits](x, act, W, y, out, ws)
            check_output(y, res, out, rows=rows)
            check_first_kernel_output(ws, L.M, L.K, bits, 128, res, rows=rows)
            del y
        del ws


@pytest.mark.parametrize("shape", [32, 16])
def test_mfma_probe_runs(shape):
    """The matrix-core probe (a measurement hook) runs on the GPU and writes
    its sink; zero operands leave every accumulator zero (without the fold)."""
    sink = B.probe_sink()
    sink.fill_(7)
    B.sq_probe_mfma_i8(3, False, False, sink, shape=shape)
    torch.cuda.synchronize()
    assert int(sink.abs().max()) == 0
    for fold in (False, True):
        B.sq_probe_mfma_i8(3, True, fold, sink, shape=shape)
        torch.cuda.synchronize()
        assert int(sink.abs().max()) > 0


@pytest.mark.parametrize("fmt", [8, 6])
def test_mfma_probe_f8f6_runs(fmt):
    """The 4-bit path's fp8 / fp6 matrix-core probe runs and writes its sink;
    zero operands leave every accumulator zero (without the fold)."""
    sink = B.probe_sink()
    sink.fill_(7)
    B.sq_probe_mfma_f8f6(fmt, 3, False, False, sink)
    torch.cuda.synchronize()
    assert int(sink.abs().max()) == 0
    for fold in (False, True):
        B.sq_probe_mfma_f8f6(fmt, 3, True, fold, sink)
        torch.cuda.synchronize()
        assert int(sink.abs().max()) > 0
