"""The allocation-free fused W4A8 linear (sq_linear_w4a8_noalloc) against the
fused linear with a caller workspace (sq_linear_w4a8): the same kernels, so
the outputs must be bit-identical; two calls in a row, the second on a smaller
layer (the scratch array keeps the first call's contents), and a layer too
large for the scratch array is refused before anything is launched."""
import ctypes

import numpy as np
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


def run_both(L, step, out):
    _, W = oracle_weight(L, 128)
    act = act_params(L, step, 8, 0)
    x = u16_to_dev(L.x_bits, torch.bfloat16)
    dt = B.OUT_DTYPES[out]
    ws = B.alloc_workspace(B.SQ_VARIANT_FUSED, L.M, L.K, L.N, 8)
    y_ref = torch.full((L.M, L.N), float("nan"), dtype=dt, device="cuda")
    B.sq_linear_w4a8(x, act, W, y_ref, out, ws)
    y = torch.full((L.M, L.N), float("nan"), dtype=dt, device="cuda")
    B.sq_linear_w4a8_noalloc(x, act, W, y, out)
    torch.cuda.synchronize()
    return y, y_ref


@pytest.mark.parametrize("out", [B.SQ_OUT_F32, B.SQ_OUT_BF16])
def test_noalloc_equals_workspace_entry(out):
    """Large then small: 2B up at 4192 tokens (tiled GEMM with a split tail,
    using the scratch array for Q_X, r and partial sums), then 300 tokens of a
    smaller layer, then 64 tokens (weight-streaming kernel with a K split)."""
    cases = [(synth.TOKENS_2B, 2048, 8192), ((200, 40, 60), 1024, 512), ((0, 0, 64), 8192, 2048)]
    for i, (tokens, K, N) in enumerate(cases):
        L = synth.make_layer(K=K, N=N, stream_counts=tokens, T=10, seed=[31, i, K, N])
        y, y_ref = run_both(L, 3 + i, out)
        assert torch.equal(y.view(torch.int16 if out != B.SQ_OUT_F32 else torch.int32),
                           y_ref.view(torch.int16 if out != B.SQ_OUT_F32 else torch.int32)), (tokens, K, N)


def test_noalloc_refuses_layers_beyond_the_scratch():
    """A layer whose fused workspace exceeds the array returns
    SQ_ERR_WORKSPACE and writes nothing; validation errors keep their codes."""
    M, K, N = 8384, 13824, 5120
    assert B.sq_workspace_bytes(B.SQ_VARIANT_FUSED, M, K, N, 8) > B.NOALLOC_SCRATCH_BYTES
    L = synth.make_layer(K=256, N=256, stream_counts=(64, 8, 16), T=2, seed=0)
    _, W = oracle_weight(L, 128)
    act = act_params(L, 0, 8, 0)
    s = act.struct()
    wt = W.struct()
    wt.K = K
    wt.N = N
    y = torch.full((4, 4), 7.0, device="cuda")
    x = torch.zeros((4, 4), dtype=torch.bfloat16, device="cuda")
    lib = B.lib()
    assert lib.sq_linear_w4a8_noalloc(x.data_ptr(), M, ctypes.byref(s), ctypes.byref(wt), y.data_ptr(),
                                      B.SQ_OUT_F32, None) == -5
    # a 4-bit activation table on the 8-bit entry point; a NULL output
    wt = W.struct()
    s4 = act_params(L, 0, 4, 0).struct()
    assert lib.sq_linear_w4a8_noalloc(x.data_ptr(), 88, ctypes.byref(s4), ctypes.byref(wt), y.data_ptr(),
                                      B.SQ_OUT_F32, None) == -4
    assert lib.sq_linear_w4a8_noalloc(x.data_ptr(), 88, ctypes.byref(s), ctypes.byref(wt), None,
                                      B.SQ_OUT_F32, None) == -1
    torch.cuda.synchronize()
    assert bool((y == 7.0).all())
