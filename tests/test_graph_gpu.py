"""The library's calls inside a captured HIP graph: every replay equals the
eager call bit for bit.  Between replays the same buffers are overwritten by
eager calls on other inputs, so a replay that reused stale workspace contents,
or a captured node that only worked the first time, would show."""
import pytest
import torch

from gpu_util import act_params, oracle_weight, u16_to_dev
from paper_2609_39056_amd import binding as B
from paper_2609_39056_amd import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.lib()


def split(M):
    a = max(M // 6, 0)
    p = max(M // 10, 0)
    return (M - a - p, p, a)


FUSED = {8: B.sq_linear_w4a8, 4: B.sq_linear_w4a4}


@pytest.mark.parametrize("bits", [8, 4])
@pytest.mark.parametrize("M,K,N,per_channel", [(64, 8192, 2048, False), (300, 2048, 512, False),
                                               (600, 1024, 384, False), (300, 2048, 512, True)])
def test_graph_replays_match_eager(bits, M, K, N, per_channel):
    """64 tokens x 8192 channels: weight-streaming kernel with a K split and
    its second kernel; 300 and 600 tokens: the tiled kernel with its split
    tail, with 128-wide weight groups or one step per output channel.  Fused
    linear and the GEMM entry point with a workspace."""
    L1 = synth.make_layer(K=K, N=N, stream_counts=split(M), T=3, seed=[11, M, K, N])
    L2 = synth.make_layer(K=K, N=N, stream_counts=split(M), T=3, seed=[12, M, K, N])
    _, W = oracle_weight(L1, K if per_channel else 128)
    x1 = u16_to_dev(L1.x_bits, torch.bfloat16)
    x2 = u16_to_dev(L2.x_bits, torch.bfloat16)
    act1, act2 = act_params(L1, 1, bits, 0), act_params(L2, 2, bits, 0)
    ws = B.alloc_workspace(B.SQ_VARIANT_FUSED, M, K, N, bits)
    wsg = B.alloc_workspace(B.SQ_VARIANT_GEMM, M, K, N, bits)
    qx, sc = B.act_buffers(M, K, bits)
    y = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
    y_gemm = torch.empty((M, N), dtype=torch.float32, device="cuda")

    def call(x, act):
        FUSED[bits](x, act, W, y, B.SQ_OUT_BF16, ws)
        B.sq_quantize_act(x, act, qx, sc)
        if bits == 8:
            B.sq_gemm_w4a8(qx, sc, W, y_gemm, B.SQ_OUT_F32, workspace=wsg)
        else:
            B.sq_gemm_w4a4(qx, sc, act, W, y_gemm, B.SQ_OUT_F32, workspace=wsg)

    call(x1, act1)
    torch.cuda.synchronize()
    ref, ref_gemm = y.clone(), y_gemm.clone()
    call(x2, act2)
    torch.cuda.synchronize()
    other = y.clone()
    assert not torch.equal(other.view(torch.int16), ref.view(torch.int16))

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        call(x1, act1)
    for rep in range(3):
        call(x2, act2)  # eager work on the same buffers between replays
        torch.cuda.synchronize()
        assert torch.equal(y.view(torch.int16), other.view(torch.int16))
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(y.view(torch.int16), ref.view(torch.int16)), f"replay {rep}"
        assert torch.equal(y_gemm.view(torch.int32), ref_gemm.view(torch.int32)), f"replay {rep}"
    del g


@pytest.mark.parametrize("bits", [8, 4])
def test_graph_calibration_replays_match_eager(bits):
    """The calibration calls captured as one HIP graph: the Eq. (9) objective
    of four candidates and a three-round constrained search (its state stays
    on the device between rounds), and the Eq. (7) objective over three
    exponents.  Every replay equals the eager results bit for bit, with eager
    calls on another layer's inputs overwriting the same workspaces between
    replays."""
    import numpy as np

    from gpu_util import f32_to_dev, i32_to_dev

    M, K, N, S = 200, 256, 128, 3
    L1 = synth.make_layer(K=K, N=N, stream_counts=split(M), T=2, seed=[13, bits])
    L2 = synth.make_layer(K=K, N=N, stream_counts=split(M), T=2, seed=[14, bits])
    _, W = oracle_weight(L1, 128)
    dev = lambda L: dict(x=u16_to_dev(L.x_bits, torch.bfloat16), t2s=i32_to_dev(L.tok2stream),
                         dinv=f32_to_dev(L.dinv), w=f32_to_dev(L.w),
                         ref=torch.empty((M, N), dtype=torch.float64, device="cuda"),
                         fp=torch.empty((M, N), dtype=torch.float64, device="cuda"))
    d1, d2 = dev(L1), dev(L2)
    gam = f32_to_dev(np.concatenate([L1.gamma, L1.gamma[::-1] * 1.1]).astype(np.float32))
    clip = f32_to_dev(np.array([L1.clip[0], L1.clip[1], L1.clip[0] * 0.8, L1.clip[1] * 1.2], np.float32))
    om = torch.full((S,), 1.0 / S, dtype=torch.float64, device="cuda")
    ws = torch.empty(max(B.sq_calib_search_workspace_bytes(M, K, N, bits, S),
                         B.sq_calib_scaling_workspace_bytes(M, K, N, 128, bits, S)), dtype=torch.uint8, device="cuda")
    obj = torch.empty(4, dtype=torch.float64, device="cuda")
    g_out = torch.empty(S, dtype=torch.float32, device="cuda")
    c_out = torch.empty(1, dtype=torch.float32, device="cuda")
    o_out = torch.empty(1, dtype=torch.float64, device="cuda")
    sobj = torch.empty(3, dtype=torch.float64, device="cuda")
    p = B.sq_calib_search_params(0.5, 2.0, float(L1.clip[0]) / 4, float(L1.clip[0]) * 4, float(L1.clip[0]), 0.5, 3)

    def call(d):
        B.sq_calib_reference(d["x"], d["dinv"], W, d["ref"])
        B.sq_calib_objective(d["x"], d["t2s"], S, d["dinv"], bits, W, d["ref"], gam, clip, om, obj, ws)
        B.sq_calib_search(d["x"], d["t2s"], S, d["dinv"], bits, W, d["ref"], om, p, g_out, c_out, o_out, ws)
        B.sq_calib_fp_reference(d["x"], d["w"], d["fp"])
        B.sq_calib_scaling_objective(d["x"], d["t2s"], S, om, d["w"], 128, bits, d["fp"], [0.25, 0.5, 0.75], sobj, ws)

    outs = lambda: [t.clone() for t in (obj, g_out, c_out, o_out, sobj)]
    call(d1)
    torch.cuda.synchronize()
    ref = outs()
    call(d2)
    torch.cuda.synchronize()
    other = outs()
    assert not torch.equal(other[0], ref[0])
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        call(d1)
    for rep in range(3):
        call(d2)
        torch.cuda.synchronize()
        assert all(torch.equal(a, b) for a, b in zip(outs(), other))
        g.replay()
        torch.cuda.synchronize()
        for a, b in zip(outs(), ref):
            assert torch.equal(a, b), f"replay {rep}"
    del g


def test_graph_chain_single_kernel_and_noalloc_replay():
    """The MLP chain with the producer-side fusion (up projection with the GELU
    epilogue, then the down projection's GEMM on its codes; and at 64 tokens,
    where the weight-streaming GEMM splits K; and with 4-bit activations, fp8
    and packed code forms), the bf16 GELU,
    the STATIC single-kernel linear (with and without a K split) and the
    allocation-free linear, captured as one HIP graph: every replay equals the
    eager calls bit for bit, with eager calls on other inputs in between."""
    Mu, K, N, N2 = 300, 2048, 1024, 256
    Lu1 = synth.make_layer(K=K, N=N, stream_counts=split(Mu), T=3, seed=[21, 1])
    Lu2 = synth.make_layer(K=K, N=N, stream_counts=split(Mu), T=3, seed=[21, 2])
    Ld = synth.make_layer(K=N, N=N2, stream_counts=split(Mu), T=3, seed=[21, 3])
    _, Wu = oracle_weight(Lu1, 128)
    _, Wd = oracle_weight(Ld, 128)
    Ms, Ks, Ns = 64, 8192, 512  # few tokens: the single-kernel linear splits K with a workspace
    Ls1 = synth.make_layer(K=Ks, N=Ns, stream_counts=(0, 0, Ms), T=3, seed=[21, 4])
    Ls2 = synth.make_layer(K=Ks, N=Ns, stream_counts=(0, 0, Ms), T=3, seed=[21, 5])
    _, Ws = oracle_weight(Ls1, 128)
    Lsd = synth.make_layer(K=Ns, N=64, stream_counts=(0, 0, Ms), T=3, seed=[21, 6])  # the few-token chain's down

    def static_act(L, step, t2s=None):
        a = act_params(L, step, 8, B.SQ_RANGE_STATIC)
        if t2s is not None:
            a.tok2stream = t2s
        return a

    xu = [u16_to_dev(L.x_bits, torch.bfloat16) for L in (Lu1, Lu2)]
    xs = [u16_to_dev(L.x_bits, torch.bfloat16) for L in (Ls1, Ls2)]
    au = [act_params(L, 1, 8, 0) for L in (Lu1, Lu2)]
    ad = [static_act(Ld, 1, au[0].tok2stream), static_act(Ld, 2, au[1].tok2stream)]
    as_ = [static_act(L, 1) for L in (Ls1, Ls2)]
    asg = [act_params(L, 1, 8, 0) for L in (Ls1, Ls2)]  # few-token chain: dynamic up projection
    asd = [static_act(Lsd, 1, asg[0].tok2stream), static_act(Lsd, 2, asg[1].tok2stream)]
    # the 4-bit chains: 300 tokens (fp8 code bytes) and 64 tokens with K split (packed codes)

    def static4(L, step, t2s):
        a = act_params(L, step, 4, B.SQ_RANGE_STATIC)
        a.tok2stream = t2s
        return a

    au4 = [act_params(L, 1, 4, 0) for L in (Lu1, Lu2)]
    ad4 = [static4(Ld, 1, au4[0].tok2stream), static4(Ld, 2, au4[1].tok2stream)]
    as4 = [act_params(L, 1, 4, 0) for L in (Ls1, Ls2)]
    asd4 = [static4(Lsd, 1, as4[0].tok2stream), static4(Lsd, 2, as4[1].tok2stream)]
    ws_u = B.alloc_workspace(B.SQ_VARIANT_FUSED, Mu, K, N, 8)
    ws_d = B.alloc_workspace(B.SQ_VARIANT_GEMM, Mu, N, N2, 8)
    ws_s = B.alloc_workspace(B.SQ_VARIANT_GEMM, Ms, Ks, Ns, 8)
    qn = torch.empty((Mu, N), dtype=torch.int8, device="cuda")
    rn = torch.empty((Mu,), dtype=torch.float32, device="cuda")
    yd = torch.empty((Mu, N2), dtype=torch.bfloat16, device="cuda")
    g_out = torch.empty((Mu, K), dtype=torch.bfloat16, device="cuda")
    ys1 = torch.empty((Ms, Ns), dtype=torch.bfloat16, device="cuda")
    ys2 = torch.empty((Ms, Ns), dtype=torch.bfloat16, device="cuda")
    yn = torch.empty((Mu, N), dtype=torch.bfloat16, device="cuda")
    ws_sg = B.alloc_workspace(B.SQ_VARIANT_FUSED, Ms, Ks, Ns, 8)
    qs = torch.empty((Ms, Ns), dtype=torch.int8, device="cuda")
    rs = torch.empty((Ms,), dtype=torch.float32, device="cuda")
    ws_u4 = B.alloc_workspace(B.SQ_VARIANT_FUSED, Mu, K, N, 4)
    q8f = torch.empty((Mu, N), dtype=torch.uint8, device="cuda")
    s8f = torch.empty((Mu, N // 64), dtype=torch.float32, device="cuda")
    k8f = torch.empty((Mu, N // 64), dtype=torch.float32, device="cuda")
    ws_s4 = B.alloc_workspace(B.SQ_VARIANT_FUSED, Ms, Ks, Ns, 4)
    q4p = torch.empty((Ms, Ns // 2), dtype=torch.uint8, device="cuda")
    s4p = torch.empty((Ms, Ns // 64), dtype=torch.float16, device="cuda")

    def call(i):
        B.sq_linear_w4a8_gelu_quant(xu[i], au[i], Wu, ad[i], qn, rn, ws_u)
        B.sq_gemm_w4a8(qn, rn, Wd, yd, B.SQ_OUT_BF16, workspace=ws_d)
        B.sq_gelu_bf16(xu[i], g_out)
        B.sq_linear_w4a8_static1(xs[i], as_[i], Ws, ys1, B.SQ_OUT_BF16)
        B.sq_linear_w4a8_static1(xs[i], as_[i], Ws, ys2, B.SQ_OUT_BF16, workspace=ws_s)
        B.sq_linear_w4a8_noalloc(xu[i], au[i], Wu, yn, B.SQ_OUT_BF16)
        B.sq_linear_w4a8_gelu_quant(xs[i], asg[i], Ws, asd[i], qs, rs, ws_sg)  # few tokens, K split
        B.sq_linear_w4a4_gelu_quant(xu[i], au4[i], Wu, ad4[i], q8f, s8f, k8f, ws_u4)
        B.sq_linear_w4a4_gelu_quant(xs[i], as4[i], Ws, asd4[i], q4p, s4p, None, ws_s4)

    outs = (qn, rn, yd, g_out, ys1, ys2, yn, qs, rs, q8f, k8f, q4p)

    def snap():
        return [t.clone() for t in outs]

    def same(a, b):
        return all(torch.equal(u.view(torch.int8), v.view(torch.int8)) for u, v in zip(a, b))

    call(0)
    torch.cuda.synchronize()
    ref = snap()
    call(1)
    torch.cuda.synchronize()
    other = snap()
    assert not any(torch.equal(u.view(torch.int8), v.view(torch.int8)) for u, v in zip(ref, other))
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        call(0)
    for rep in range(3):
        call(1)
        torch.cuda.synchronize()
        assert same(snap(), other)
        g.replay()
        torch.cuda.synchronize()
        assert same(snap(), ref), f"replay {rep}"
    del g
