"""Hand-derived worked cases of the quantizers (tests/golden/quantize_worked_cases.json):
every input is a small dyadic rational, so each expected code and step follows
from Eq. 1 (with Eq. 6's channel scaling and Eq. 8's stream gain) by
inspection, independently of any program.  The oracle must reproduce them
(CPU), and so must the HIP quantizer and weight packer (GPU)."""
import json
import os

import numpy as np
import pytest

from oracle import sq_oracle as O

HERE = os.path.dirname(os.path.abspath(__file__))
CASES = json.load(open(os.path.join(HERE, "golden", "quantize_worked_cases.json")))
MODE = {"dynamic": O.RANGE_DYNAMIC, "static": O.RANGE_STATIC}


def padded(vals, n):
    out = np.zeros(n, dtype=np.float32)
    out[:len(vals)] = vals
    return out


def activation_inputs(case):
    """bf16 bits [M, K], stream map, gain table, D^-1 (ones past the listed
    channels, or None), thresholds, and the expected codes / steps."""
    K, bits = case["K"], case["act_bits"]
    rows = case["rows"]
    x = np.zeros((len(rows), K), dtype=np.float32)
    codes = np.zeros((len(rows), K), dtype=np.int64)
    for i, r in enumerate(rows):
        if bits == 8:
            x[i] = padded(r["x"], K)
            codes[i] = padded(r["codes"], K)
        else:
            x[i, :64] = padded(r["x"], 64)
            x[i, 64:] = padded(r["x_group1"], 64)
            codes[i, :64] = padded(r["codes"], 64)
            codes[i, 64:] = padded(r["codes_group1"], 64)
    x_bits = O.f32_to_bf16_bits(x)
    assert np.array_equal(O.bf16_bits_to_f32(x_bits), x), "inputs must be exact in bf16"
    t2s = np.array([r["stream"] for r in rows], dtype=np.int32)
    gamma = np.array(case["gamma"], dtype=np.float32)
    dinv = padded(case["dinv"], K) if "dinv" in case else None
    if dinv is not None:
        dinv[len(case["dinv"]):] = 1.0
    clip = np.array(case["clip"], dtype=np.float32) if "clip" in case else np.ones(gamma.shape[0], np.float32)
    if bits == 8:
        steps = np.array([r["scale"] for r in rows], dtype=np.float32)
    else:
        steps = np.array([r["group_steps"] for r in rows], dtype=np.float32)
    return x_bits, t2s, gamma, dinv, clip, codes, steps


def weight_inputs(case):
    K, G = case["K"], case["w_group"]
    assert K == 2 * G
    rows = case["rows"]
    w = np.zeros((len(rows), K), dtype=np.float32)
    codes = np.zeros((len(rows), K), dtype=np.int64)
    for i, r in enumerate(rows):
        w[i, :G] = padded(r["w"], G)
        w[i, G:] = padded(r["w_group1"], G)
        codes[i, :G] = padded(r["codes"], G)
        codes[i, G:] = padded(r["codes_group1"], G)
    steps = np.array([r["steps"] for r in rows], dtype=np.float32)
    return w, codes, steps


@pytest.mark.parametrize("case", CASES["activation_cases"], ids=lambda c: c["name"])
def test_oracle_quantizer_worked_cases(case):
    x_bits, t2s, gamma, dinv, clip, codes, steps = activation_inputs(case)
    ref = O.quantize_act(x_bits, t2s, gamma, case["step"], dinv=dinv, clip=clip,
                         range_mode=MODE[case["range_mode"]], act_bits=case["act_bits"])
    assert np.array_equal(ref["codes"].astype(np.int64), codes)
    if case["act_bits"] == 8:
        assert np.array_equal(ref["scale"], steps)
    else:
        assert np.array_equal(O.f16_bits_to_f32(ref["scale"]), steps)


@pytest.mark.parametrize("case", CASES["weight_cases"], ids=lambda c: c["name"])
def test_oracle_weight_packing_worked_cases(case):
    w, codes, steps = weight_inputs(case)
    ref = O.pack_weights(w, None, case["w_group"])
    assert np.array_equal(ref["codes"].astype(np.int64), codes)
    assert np.array_equal(O.f16_bits_to_f32(ref["w_scale"]), steps)


@pytest.mark.gpu
@pytest.mark.parametrize("case", CASES["activation_cases"], ids=lambda c: c["name"])
def test_gpu_quantizer_worked_cases(case):
    import torch

    from gpu_util import f32_to_dev, i32_to_dev, u16_to_dev
    from paper_2609_39056_amd import binding as B

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    x_bits, t2s, gamma, dinv, clip, codes, steps = activation_inputs(case)
    M, K, bits = x_bits.shape[0], case["K"], case["act_bits"]
    act = B.ActParams(tok2stream=i32_to_dev(t2s), gamma=f32_to_dev(gamma), step=case["step"], act_bits=bits,
                      range_mode=MODE[case["range_mode"]], clip=f32_to_dev(clip),
                      dinv=None if dinv is None else f32_to_dev(dinv))
    qx, sc = B.act_buffers(M, K, bits)
    B.sq_quantize_act(u16_to_dev(x_bits, torch.bfloat16), act, qx, sc)
    torch.cuda.synchronize()
    if bits == 8:
        assert np.array_equal(qx.cpu().numpy().astype(np.int64), codes)
        assert np.array_equal(sc.cpu().numpy(), steps)
    else:
        assert np.array_equal(qx.cpu().numpy(), O.pack_int4(codes.astype(np.int8)))
        assert np.array_equal(sc.cpu().float().numpy(), steps)


@pytest.mark.gpu
@pytest.mark.parametrize("case", CASES["weight_cases"], ids=lambda c: c["name"])
def test_gpu_weight_packing_worked_cases(case):
    import torch

    from gpu_util import f32_to_dev
    from paper_2609_39056_amd import binding as B

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    w, codes, steps = weight_inputs(case)
    n = w.shape[0]
    # the library takes N in multiples of 64: zero rows after the worked ones
    # (their codes and steps are 0)
    wp = np.zeros((64, w.shape[1]), dtype=np.float32)
    wp[:n] = w
    W = B.prepare_weight(f32_to_dev(wp), None, case["w_group"])
    torch.cuda.synchronize()
    qw = W.qw.cpu().numpy()
    assert np.array_equal(qw[:n], O.pack_int4(codes.astype(np.int8)))
    assert not qw[n:].any()
    # the device stores the steps group-major: [K / w_group][N]
    ws = W.w_scale.cpu().float().numpy().T
    assert np.array_equal(ws[:n], steps)
    assert not ws[n:].any()
