"""Helpers for the GPU parity tests: moving seeded inputs to the device and
the comparison rules (bit-exact integers, fp32 within 1e-5 of the summation
scale, bf16 / fp16 within 1 ulp)."""
import numpy as np
import torch

from oracle import sq_oracle as O
from paper_2609_39056_amd import binding as B

DEV = "cuda"


def u16_to_dev(bits, dtype):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(dtype).to(DEV)


def f32_to_dev(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(DEV)


def i32_to_dev(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(DEV)


def u8_to_dev(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.uint8)).to(DEV)


def bits16(t):
    """Device fp16 / bf16 tensor -> host uint16 bit patterns."""
    return t.detach().cpu().view(torch.int16).numpy().view(np.uint16)


def act_params(L, step, act_bits=8, range_mode=B.SQ_RANGE_DYNAMIC, use_dinv=True, rows=None):
    t2s = L.tok2stream if rows is None else L.tok2stream[rows]
    return B.ActParams(
        tok2stream=i32_to_dev(t2s), gamma=f32_to_dev(L.gamma), step=step, act_bits=act_bits,
        range_mode=range_mode, clip=f32_to_dev(L.clip), dinv=f32_to_dev(L.dinv) if use_dinv else None)


def oracle_weight(L, w_group, with_bias=True):
    """Weights prepared by the oracle, as device tensors (inputs to the HIP path)."""
    pw = O.pack_weights(L.w, L.d, w_group)
    # the C ABI stores weight steps group-major: [K/w_group][N]
    dev = B.Weight(qw=u8_to_dev(pw["qw"]), w_scale=u16_to_dev(pw["w_scale"].T, torch.float16),
                   w_group=w_group,
                   bias=u16_to_dev(L.bias_bits, torch.bfloat16) if with_bias else None)
    return pw, dev


def ordered16(bits):
    """uint16 float bit patterns -> integers ordered like the values (+0 == -0)."""
    b = bits.astype(np.int64)
    return np.where(b & 0x8000, -(b & 0x7FFF), b)


def check_output(y_dev, res, out_dtype, rows=None):
    """Compare a device output with the oracle result dict (canonical fp32 y,
    and A = sum of |terms|)."""
    y_or = res["y"]
    A = res["A"]
    if rows is not None:
        y_dev = y_dev[torch.as_tensor(rows, device=y_dev.device)]
    if out_dtype == B.SQ_OUT_F32:
        y = y_dev.cpu().numpy().astype(np.float64)
        err = np.abs(y - y_or.astype(np.float64))
        assert np.all(err <= 1e-5 * A), f"max err/A = {np.max(err / np.maximum(A, 1e-300))}"
        # element-relative where the sum keeps a tenth of its magnitude: there
        # 1e-5 |y| >= 1e-6 A, about 17 units of 2^-24 A, several times what a
        # different summation order of the blocks costs
        nc = np.abs(y_or) >= 0.1 * A
        if nc.any():
            rel = err[nc] / np.abs(y_or[nc].astype(np.float64))
            assert rel.max() <= 1e-5, f"max rel = {rel.max()}"
        return float(np.max(err / np.maximum(A, 1e-300)))
    fmt = "bf16" if out_dtype == B.SQ_OUT_BF16 else "f16"
    want = O.cast_output(y_or, fmt)
    got = bits16(y_dev)
    d = np.abs(ordered16(got) - ordered16(want))
    # 1 ulp where the sum does not cancel; where it does (|y| < A/100) the
    # fp32 results may legitimately differ by 1e-5 * A, which is many ulps of
    # a tiny y: there the cast value must lie within 1e-5 * A + 1 ulp of y.
    nc = np.abs(y_or) >= 0.01 * A
    assert d[nc].max(initial=0) <= 1, f"max ulp diff (non-cancelling) {d[nc].max()}"
    to32 = O.bf16_bits_to_f32 if fmt == "bf16" else O.f16_bits_to_f32
    gv = to32(got).astype(np.float64)
    wv = to32(want).astype(np.float64)
    last_finite = 0x7F7F if fmt == "bf16" else 0x7BFF
    step = np.where((want & 0x7FFF) < last_finite, want.astype(np.int64) + 1, want.astype(np.int64) - 1)
    ulp = np.abs(to32(step.astype(np.uint16)).astype(np.float64) - wv)
    err = np.abs(gv - y_or.astype(np.float64))
    assert np.all(err <= 1e-5 * A + ulp), "cast output outside 1e-5*A + 1 ulp"
    return int(d[nc].max(initial=0))


def _align(n):
    return (n + 255) // 256 * 256


def fused_first_kernel_output(ws, M, K, bits, w_group, rows=None):
    """What the fused linear's first kernel left in its workspace (the layout
    include/sq.h documents), for `rows` (default all): the codes as int
    [rows, K], the scales as raw bits (uint32 r, or uint16 sigma [rows, K/64];
    the fp8 path stores sigma as fp32, returned as its fp16 bits) and, for
    4-bit codes on the fp8 path, kc as fp32 [rows, K/64] (else None).
    Rows are selected on the device."""
    ri = None if rows is None else torch.as_tensor(np.asarray(rows, dtype=np.int64), device=ws.device)
    pick = (lambda t: t) if ri is None else (lambda t: t[ri])
    if bits == 8:
        codes = pick(ws[: M * K].view(M, K)).cpu().numpy().view(np.int8).astype(np.int64)
        off = _align(M * K)
        r = pick(ws[off: off + 4 * M].view(torch.int32)).cpu().numpy().view(np.uint32)
        return codes, r, None
    f8 = M > 128  # more than 128 tokens: the fp8 path (include/sq.h)
    g = K // 64
    if f8:
        b = pick(ws[: M * K].view(M, K)).cpu().numpy().astype(np.int64)
        codes = np.where(b & 0x80, -(b & 0x7F), b & 0x7F)
        off = _align(M * K)
    else:
        packed = pick(ws[: M * K // 2].view(M, K // 2)).cpu().numpy()
        codes = O.unpack_int4(packed).astype(np.int64)
        off = _align(M * K // 2)
    kc = None
    if f8:  # fp32 steps (the fp16 values widened), then kc
        s32 = pick(ws[off: off + 4 * M * g].view(torch.float32).view(M, g)).cpu().numpy()
        sigma = s32.astype(np.float16).view(np.uint16)
        assert np.array_equal(sigma.view(np.float16).astype(np.float32), s32), "steps not fp16 values"
        off += _align(4 * M * g)
        kc = pick(ws[off: off + 4 * M * g].view(torch.float32).view(M, g)).cpu().numpy()
    else:
        sigma = pick(ws[off: off + 2 * M * g].view(torch.int16).view(M, g)).cpu().numpy().view(np.uint16)
    return codes, sigma, kc


def check_first_kernel_output(ws, M, K, bits, w_group, res, rows=None):
    """Codes and stored scales bit-exact against the oracle's quantize step
    (res: O.linear's result for the same rows); fp8 4-bit path: kc too."""
    codes, sc, kc = fused_first_kernel_output(ws, M, K, bits, w_group, rows)
    assert np.array_equal(codes, res["codes"].astype(np.int64))
    if bits == 8:
        assert np.array_equal(sc, np.asarray(res["scale"], dtype=np.float32).view(np.uint32))
    else:
        assert np.array_equal(sc, np.asarray(res["scale"]).view(np.uint16))
        if kc is not None:  # values exact (a zero sum may give either sign of zero)
            assert np.array_equal(kc, expected_kc(codes, sc))


def expected_kc(codes, sigma_bits):
    """-8 * S * sigma * 2^-18 per (row, 64-group), S the group's code sum
    (exact in fp32: |8 S| < 2^12 and sigma has an 11-bit significand)."""
    M, K = codes.shape
    S = codes.reshape(M, K // 64, 64).sum(axis=2)
    sig = sigma_bits.view(np.float16).astype(np.float64)
    return (-8.0 * S * sig * 2.0 ** -18).astype(np.float32)
