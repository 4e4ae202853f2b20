"""ctypes binding of libsq (include/sq.h).  Argument marshalling only: every
step of the linear runs in the HIP kernels of the library.

The functions carry the C names.  Device buffers are torch tensors on the GPU
(torch supplies the memory and the stream); shapes are read from them.  A
non-zero status raises SqError.  If the library has not been built, loading
fails loudly: there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional

import torch

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "lib", "libsq.so")

SQ_OK = 0
SQ_RANGE_DYNAMIC = 0
SQ_RANGE_STATIC = 1
SQ_OUT_F32 = 0
SQ_OUT_BF16 = 1
SQ_OUT_F16 = 2
SQ_VARIANT_FUSED = 0
SQ_VARIANT_UNFUSED = 1
SQ_VARIANT_GEMM = 2
A4_GROUP = 64

OUT_DTYPES = {SQ_OUT_F32: torch.float32, SQ_OUT_BF16: torch.bfloat16, SQ_OUT_F16: torch.float16}


class SqError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"{what}: {status_string(status)} ({status})")
        self.status = status


class sq_act_params(ctypes.Structure):
    _fields_ = [
        ("tok2stream", ctypes.c_void_p),
        ("gamma", ctypes.c_void_p),
        ("clip", ctypes.c_void_p),
        ("dinv", ctypes.c_void_p),
        ("num_streams", ctypes.c_int32),
        ("num_steps", ctypes.c_int32),
        ("step", ctypes.c_int32),
        ("range_mode", ctypes.c_int32),
        ("act_bits", ctypes.c_int32),
    ]


class sq_weight(ctypes.Structure):
    _fields_ = [
        ("qw", ctypes.c_void_p),
        ("w_scale", ctypes.c_void_p),
        ("bias", ctypes.c_void_p),
        ("N", ctypes.c_int32),
        ("K", ctypes.c_int32),
        ("w_group", ctypes.c_int32),
    ]


class sq_calib_search_params(ctypes.Structure):
    _fields_ = [
        ("gamma_min", ctypes.c_float),
        ("gamma_max", ctypes.c_float),
        ("clip_min", ctypes.c_float),
        ("clip_max", ctypes.c_float),
        ("clip_init", ctypes.c_float),
        ("log_step", ctypes.c_float),
        ("rounds", ctypes.c_int32),
    ]


_P = ctypes.c_void_p
_I = ctypes.c_int32
_S = ctypes.c_size_t
_SIGS = {
    "sq_status_string": (ctypes.c_char_p, [_I]),
    "sq_workspace_bytes": (_S, [_I, _I, _I, _I, _I]),
    "sq_pack_weights": (_I, [_P, _P, _I, _I, _I, _P, _P, _P]),
    "sq_quantize_act": (_I, [_P, _I, _I, ctypes.POINTER(sq_act_params), _P, _P, _P]),
    "sq_gemm_w4a8": (_I, [_P, _P, _I, ctypes.POINTER(sq_weight), _P, _I, _P, _S, _P]),
    "sq_gemm_w4a4": (_I, [_P, _P, _I, ctypes.POINTER(sq_act_params), ctypes.POINTER(sq_weight), _P, _I, _P, _S,
                          _P]),
    "sq_linear_w4a8": (_I, [_P, _I, ctypes.POINTER(sq_act_params), ctypes.POINTER(sq_weight), _P, _I, _P, _S, _P]),
    "sq_linear_w4a4": (_I, [_P, _I, ctypes.POINTER(sq_act_params), ctypes.POINTER(sq_weight), _P, _I, _P, _S, _P]),
    "sq_linear_unfused": (_I, [_P, _I, ctypes.POINTER(sq_act_params), ctypes.POINTER(sq_weight), _P, _I, _P, _S, _P]),
    "sq_linear_w4a8_noalloc": (_I, [_P, _I, ctypes.POINTER(sq_act_params), ctypes.POINTER(sq_weight), _P, _I, _P]),
    "sq_linear_w4a8_static1": (_I, [_P, _I, ctypes.POINTER(sq_act_params), ctypes.POINTER(sq_weight), _P, _I, _P, _S,
                                    _P]),
    "sq_linear_w4a8_gelu_quant": (_I, [_P, _I, ctypes.POINTER(sq_act_params), ctypes.POINTER(sq_weight),
                                       ctypes.POINTER(sq_act_params), _P, _P, _P, _S, _P]),
    "sq_linear_w4a4_gelu_quant": (_I, [_P, _I, ctypes.POINTER(sq_act_params), ctypes.POINTER(sq_weight),
                                       ctypes.POINTER(sq_act_params), _P, _P, _P, _P, _S, _P]),
    "sq_gemm_w4a4_fp8": (_I, [_P, _P, _P, _I, ctypes.POINTER(sq_act_params), ctypes.POINTER(sq_weight), _P, _I, _P,
                              _S, _P]),
    "sq_gelu_bf16": (_I, [_P, _S, _P, _P]),
    "sq_debug_block_acc_i32": (_I, [_P, _I, _I, ctypes.POINTER(sq_weight), _P, _P]),
    "sq_calib_reference": (_I, [_P, _I, _P, ctypes.POINTER(sq_weight), _P, _P]),
    "sq_calib_workspace_bytes": (_S, [_I, _I, _I, _I, _I]),
    "sq_calib_objective": (_I, [_P, _I, _P, _I, _P, _I, ctypes.POINTER(sq_weight), _P, _I, _P, _P, _P, _P, _P, _S,
                                _P]),
    "sq_calib_fp_reference": (_I, [_P, _I, _P, _I, _I, _P, _P]),
    "sq_smooth_scales": (_I, [_P, _I, _P, _I, _I, ctypes.c_float, _P, _P, _P]),
    "sq_calib_scaling_workspace_bytes": (_S, [_I, _I, _I, _I, _I, _I]),
    "sq_calib_scaling_objective": (_I, [_P, _I, _P, _I, _P, _P, _I, _I, _I, _I, _P, _I,
                                        ctypes.POINTER(ctypes.c_float), _P, _P, _S, _P]),
    "sq_calib_search_workspace_bytes": (_S, [_I, _I, _I, _I, _I]),
    "sq_calib_search": (_I, [_P, _I, _P, _I, _P, _I, ctypes.POINTER(sq_weight), _P, _P,
                             ctypes.POINTER(sq_calib_search_params), _P, _P, _P, _P, _S, _P]),
    "sq_probe_mfma_i8_sink_bytes": (_S, []),
    "sq_probe_mfma_i8": (_I, [_I, _I, _I, _I, _P, _S, _P]),
    "sq_probe_mfma_f8f6": (_I, [_I, _I, _I, _I, _P, _S, _P]),
}

_lib = None


def lib() -> ctypes.CDLL:
    """Load libsq.so (built by paper_2609_39056_amd._build) and declare its
    signatures.  Raises if the library is missing."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} not found: build it first (python -m paper_2609_39056_amd._build)")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def status_string(status: int) -> str:
    return lib().sq_status_string(int(status)).decode()


def _check(status: int, what: str) -> None:
    if status != SQ_OK:
        raise SqError(status, what)


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("libsq takes device tensors")
    if not t.is_contiguous():
        raise ValueError("libsq takes contiguous tensors")
    return t.data_ptr()


def _stream(stream) -> int:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


@dataclass
class ActParams:
    """Device tensors of the activation-side table for one layer."""

    tok2stream: torch.Tensor           # int32 [M]
    gamma: torch.Tensor                # fp32 [T, S]
    step: int
    act_bits: int = 8
    range_mode: int = SQ_RANGE_DYNAMIC
    clip: Optional[torch.Tensor] = None  # fp32 [T]
    dinv: Optional[torch.Tensor] = None  # fp32 [K]

    def struct(self) -> sq_act_params:
        T, S = self.gamma.shape
        return sq_act_params(_ptr(self.tok2stream), _ptr(self.gamma), _ptr(self.clip), _ptr(self.dinv),
                             S, T, self.step, self.range_mode, self.act_bits)


@dataclass
class Weight:
    """A prepared int4 weight on the device."""

    qw: torch.Tensor                   # uint8 [N, K/2]
    w_scale: torch.Tensor              # fp16 [K/w_group, N], group-major
    w_group: int
    bias: Optional[torch.Tensor] = None  # bf16 [N]

    @property
    def N(self) -> int:
        return int(self.qw.shape[0])

    @property
    def K(self) -> int:
        return int(self.qw.shape[1]) * 2

    def struct(self) -> sq_weight:
        return sq_weight(_ptr(self.qw), _ptr(self.w_scale), _ptr(self.bias), self.N, self.K, self.w_group)


def sq_workspace_bytes(variant: int, M: int, K: int, N: int, act_bits: int) -> int:
    return int(lib().sq_workspace_bytes(variant, M, K, N, act_bits))


def sq_pack_weights(w: torch.Tensor, d: Optional[torch.Tensor], w_group: int, qw: torch.Tensor,
                    w_scale: torch.Tensor, stream=None) -> None:
    N, K = w.shape
    _check(lib().sq_pack_weights(_ptr(w), _ptr(d), N, K, w_group, _ptr(qw), _ptr(w_scale), _stream(stream)),
           "sq_pack_weights")


def sq_quantize_act(x: torch.Tensor, act: ActParams, qx: torch.Tensor, act_scale: torch.Tensor,
                    stream=None) -> None:
    M, K = x.shape
    s = act.struct()
    _check(lib().sq_quantize_act(_ptr(x), M, K, ctypes.byref(s), _ptr(qx), _ptr(act_scale), _stream(stream)),
           "sq_quantize_act")


def _ws(workspace: Optional[torch.Tensor]):
    if workspace is None:
        return None, 0
    return _ptr(workspace), workspace.numel() * workspace.element_size()


def sq_gemm_w4a8(qx: torch.Tensor, row_scale: torch.Tensor, w: Weight, y: torch.Tensor, out_dtype: int,
                 workspace: Optional[torch.Tensor] = None, stream=None) -> None:
    M = qx.shape[0]
    ws = w.struct()
    wp, wb = _ws(workspace)
    _check(lib().sq_gemm_w4a8(_ptr(qx), _ptr(row_scale), M, ctypes.byref(ws), _ptr(y), out_dtype, wp, wb,
                              _stream(stream)), "sq_gemm_w4a8")


def sq_gemm_w4a4(qx: torch.Tensor, group_scale: torch.Tensor, act: ActParams, w: Weight, y: torch.Tensor,
                 out_dtype: int, workspace: Optional[torch.Tensor] = None, stream=None) -> None:
    M = qx.shape[0]
    s, ws = act.struct(), w.struct()
    wp, wb = _ws(workspace)
    _check(lib().sq_gemm_w4a4(_ptr(qx), _ptr(group_scale), M, ctypes.byref(s), ctypes.byref(ws), _ptr(y),
                              out_dtype, wp, wb, _stream(stream)), "sq_gemm_w4a4")


def _linear(fn: str, x, act, w, y, out_dtype, workspace, stream):
    M = x.shape[0]
    s, ws = act.struct(), w.struct()
    st = getattr(lib(), fn)(_ptr(x), M, ctypes.byref(s), ctypes.byref(ws), _ptr(y), out_dtype,
                            _ptr(workspace), workspace.numel() * workspace.element_size(), _stream(stream))
    _check(st, fn)


def sq_linear_w4a8(x, act: ActParams, w: Weight, y, out_dtype: int, workspace, stream=None) -> None:
    _linear("sq_linear_w4a8", x, act, w, y, out_dtype, workspace, stream)


def sq_linear_w4a4(x, act: ActParams, w: Weight, y, out_dtype: int, workspace, stream=None) -> None:
    _linear("sq_linear_w4a4", x, act, w, y, out_dtype, workspace, stream)


def sq_linear_w4a8_static1(x, act: ActParams, w: Weight, y, out_dtype: int, workspace=None, stream=None) -> None:
    """The STATIC single-kernel W4A8 linear for at most 128 tokens (include/sq.h);
    workspace None (no K split) or a SQ_VARIANT_GEMM workspace."""
    M = x.shape[0]
    s, ws = act.struct(), w.struct()
    nbytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().sq_linear_w4a8_static1(_ptr(x), M, ctypes.byref(s), ctypes.byref(ws), _ptr(y), out_dtype,
                                        _ptr(workspace), nbytes, _stream(stream)), "sq_linear_w4a8_static1")


def sq_linear_w4a8_gelu_quant(x, act: ActParams, w: Weight, act_next: ActParams, qx_next, r_next, workspace,
                              stream=None) -> None:
    """The up projection with the GELU epilogue that writes the down
    projection's STATIC codes qx_next (int8 [M, N]) and row scales r_next
    (fp32 [M]) (include/sq.h); workspace as for sq_linear_w4a8."""
    M = x.shape[0]
    s, ws, sn = act.struct(), w.struct(), act_next.struct()
    _check(lib().sq_linear_w4a8_gelu_quant(_ptr(x), M, ctypes.byref(s), ctypes.byref(ws), ctypes.byref(sn),
                                           _ptr(qx_next), _ptr(r_next), _ptr(workspace),
                                           workspace.numel() * workspace.element_size(), _stream(stream)),
           "sq_linear_w4a8_gelu_quant")


def sq_linear_w4a4_gelu_quant(x, act: ActParams, w: Weight, act_next: ActParams, qx_next, scale_next, kc_next,
                              workspace, stream=None) -> None:
    """The W4A4 up projection with the GELU epilogue that writes the down
    projection's STATIC 4-bit codes (include/sq.h): at most 128 tokens packed
    int4 qx_next [M, N/2] and fp16 scale_next [M, N/64] (kc_next None);
    more, fp8 code bytes qx_next [M, N] with fp32 scale_next and kc_next
    [M, N/64].  workspace as for sq_linear_w4a4."""
    M = x.shape[0]
    s, ws, sn = act.struct(), w.struct(), act_next.struct()
    _check(lib().sq_linear_w4a4_gelu_quant(_ptr(x), M, ctypes.byref(s), ctypes.byref(ws), ctypes.byref(sn),
                                           _ptr(qx_next), _ptr(scale_next), _ptr(kc_next), _ptr(workspace),
                                           workspace.numel() * workspace.element_size(), _stream(stream)),
           "sq_linear_w4a4_gelu_quant")


def sq_gemm_w4a4_fp8(qx, group_scale, kc, act: ActParams, w: Weight, y, out_dtype: int, workspace=None,
                     stream=None) -> None:
    """The 4-bit GEMM on fp8 code bytes [M, K] with fp32 group steps and kc
    [M, K/64] (more than 128 tokens; include/sq.h)."""
    M = qx.shape[0]
    s, ws = act.struct(), w.struct()
    wp, wb = _ws(workspace)
    _check(lib().sq_gemm_w4a4_fp8(_ptr(qx), _ptr(group_scale), _ptr(kc), M, ctypes.byref(s), ctypes.byref(ws),
                                  _ptr(y), out_dtype, wp, wb, _stream(stream)), "sq_gemm_w4a4_fp8")


def sq_gelu_bf16(x, y, stream=None) -> None:
    """y = bf16 GELU of the bf16 tensor x (same number of elements; y may be x)."""
    n = x.numel()
    assert y.numel() == n
    _check(lib().sq_gelu_bf16(_ptr(x), n, _ptr(y), _stream(stream)), "sq_gelu_bf16")


def sq_linear_unfused(x, act: ActParams, w: Weight, y, out_dtype: int, workspace, stream=None) -> None:
    _linear("sq_linear_unfused", x, act, w, y, out_dtype, workspace, stream)


NOALLOC_SCRATCH_BYTES = 64 << 20  # SQ_NOALLOC_SCRATCH_BYTES


def sq_linear_w4a8_noalloc(x, act: ActParams, w: Weight, y, out_dtype: int, stream=None) -> None:
    """sq_linear_w4a8 without a workspace argument: the library's own device
    scratch array holds Q_X, r and the partial sums (include/sq.h)."""
    s, ws = act.struct(), w.struct()
    _check(lib().sq_linear_w4a8_noalloc(_ptr(x), x.shape[0], ctypes.byref(s), ctypes.byref(ws), _ptr(y), out_dtype,
                                        _stream(stream)), "sq_linear_w4a8_noalloc")


def sq_debug_block_acc_i32(qx: torch.Tensor, act_bits: int, w: Weight, acc_out: torch.Tensor,
                           stream=None) -> None:
    M = qx.shape[0]
    ws = w.struct()
    _check(lib().sq_debug_block_acc_i32(_ptr(qx), M, act_bits, ctypes.byref(ws), _ptr(acc_out),
                                        _stream(stream)), "sq_debug_block_acc_i32")


def sq_calib_reference(x: torch.Tensor, dinv: Optional[torch.Tensor], w: Weight, y_ref: torch.Tensor,
                       stream=None) -> None:
    """The Eq. (9) target X~ W^ into fp64 y_ref [M, N] (include/sq.h)."""
    M = x.shape[0]
    ws = w.struct()
    _check(lib().sq_calib_reference(_ptr(x), M, _ptr(dinv), ctypes.byref(ws), _ptr(y_ref), _stream(stream)),
           "sq_calib_reference")


def sq_calib_workspace_bytes(M: int, K: int, N: int, act_bits: int, num_streams: int) -> int:
    return int(lib().sq_calib_workspace_bytes(M, K, N, act_bits, num_streams))


def sq_calib_objective(x: torch.Tensor, tok2stream: torch.Tensor, num_streams: int, dinv: Optional[torch.Tensor],
                       act_bits: int, w: Weight, y_ref: torch.Tensor, cand_gamma: torch.Tensor,
                       cand_clip: torch.Tensor, omega: torch.Tensor, objective: torch.Tensor,
                       workspace: torch.Tensor, stream=None) -> None:
    """Eq. (9) for every candidate row of cand_gamma [C, S] / cand_clip [C]
    into fp64 objective [C] (include/sq.h)."""
    M = x.shape[0]
    C = cand_clip.shape[0]
    ws = w.struct()
    wp, wb = _ws(workspace)
    _check(lib().sq_calib_objective(_ptr(x), M, _ptr(tok2stream), num_streams, _ptr(dinv), act_bits,
                                    ctypes.byref(ws), _ptr(y_ref), C, _ptr(cand_gamma), _ptr(cand_clip),
                                    _ptr(omega), _ptr(objective), wp, wb, _stream(stream)), "sq_calib_objective")


def sq_calib_fp_reference(x: torch.Tensor, w: torch.Tensor, y_ref: torch.Tensor, stream=None) -> None:
    """The full-precision target X W^T of Eq. (7) into fp64 y_ref [M, N]."""
    M, K = x.shape
    N = w.shape[0]
    _check(lib().sq_calib_fp_reference(_ptr(x), M, _ptr(w), N, K, _ptr(y_ref), _stream(stream)),
           "sq_calib_fp_reference")


def sq_smooth_scales(x: torch.Tensor, w: torch.Tensor, alpha: float, d: torch.Tensor, dinv: torch.Tensor,
                     stream=None) -> None:
    """d = amax|X|^alpha / amax|W|^(1 - alpha) per channel (clamped) and 1 / d."""
    M, K = x.shape
    N = w.shape[0]
    _check(lib().sq_smooth_scales(_ptr(x), M, _ptr(w), N, K, float(alpha), _ptr(d), _ptr(dinv), _stream(stream)),
           "sq_smooth_scales")


def sq_calib_scaling_workspace_bytes(M: int, K: int, N: int, w_group: int, act_bits: int, num_regions: int) -> int:
    return int(lib().sq_calib_scaling_workspace_bytes(M, K, N, w_group, act_bits, num_regions))


def sq_calib_scaling_objective(x: torch.Tensor, region: torch.Tensor, num_regions: int, region_weight: torch.Tensor,
                               w: torch.Tensor, w_group: int, act_bits: int, y_ref: torch.Tensor, alphas,
                               objective: torch.Tensor, workspace: torch.Tensor, stream=None) -> None:
    """Eq. (7) for each exponent in `alphas` (a host sequence) into fp64 objective."""
    M, K = x.shape
    N = w.shape[0]
    a = (ctypes.c_float * len(alphas))(*[float(v) for v in alphas])
    wp, wb = _ws(workspace)
    _check(lib().sq_calib_scaling_objective(_ptr(x), M, _ptr(region), num_regions, _ptr(region_weight), _ptr(w), N,
                                            K, w_group, act_bits, _ptr(y_ref), len(alphas), a, _ptr(objective), wp,
                                            wb, _stream(stream)), "sq_calib_scaling_objective")


def sq_calib_search_workspace_bytes(M: int, K: int, N: int, act_bits: int, num_streams: int) -> int:
    return int(lib().sq_calib_search_workspace_bytes(M, K, N, act_bits, num_streams))


def sq_calib_search(x: torch.Tensor, tok2stream: torch.Tensor, num_streams: int, dinv: Optional[torch.Tensor],
                    act_bits: int, w: Weight, y_ref: torch.Tensor, omega: torch.Tensor,
                    params: sq_calib_search_params, gamma_out: torch.Tensor, clip_out: torch.Tensor,
                    objective_out: torch.Tensor, workspace: torch.Tensor, stream=None) -> None:
    """Constrained compass search for Eq. (9)'s (gamma*, c*) (include/sq.h)."""
    M = x.shape[0]
    ws = w.struct()
    wp, wb = _ws(workspace)
    _check(lib().sq_calib_search(_ptr(x), M, _ptr(tok2stream), num_streams, _ptr(dinv), act_bits, ctypes.byref(ws),
                                 _ptr(y_ref), _ptr(omega), ctypes.byref(params), _ptr(gamma_out), _ptr(clip_out),
                                 _ptr(objective_out), wp, wb, _stream(stream)), "sq_calib_search")


# ------------------------------------------------------------------ helpers
def alloc_workspace(variant: int, M: int, K: int, N: int, act_bits: int, device="cuda") -> torch.Tensor:
    n = sq_workspace_bytes(variant, M, K, N, act_bits)
    if n == 0:
        raise ValueError("invalid shape for workspace")
    return torch.empty(n, dtype=torch.uint8, device=device)


def prepare_weight(w: torch.Tensor, d: Optional[torch.Tensor], w_group: int,
                   bias: Optional[torch.Tensor] = None, stream=None) -> Weight:
    """Fold, quantize and pack a device fp32 weight [N, K] with sq_pack_weights."""
    N, K = w.shape
    qw = torch.empty((N, K // 2), dtype=torch.uint8, device=w.device)
    ws = torch.empty((K // w_group, N), dtype=torch.float16, device=w.device)
    sq_pack_weights(w, d, w_group, qw, ws, stream)
    return Weight(qw=qw, w_scale=ws, w_group=w_group, bias=bias)


def act_buffers(M: int, K: int, act_bits: int, device="cuda"):
    """Allocate Q_X and its scales for sq_quantize_act."""
    if act_bits == 8:
        return (torch.empty((M, K), dtype=torch.int8, device=device),
                torch.empty((M,), dtype=torch.float32, device=device))
    return (torch.empty((M, K // 2), dtype=torch.uint8, device=device),
            torch.empty((M, K // A4_GROUP), dtype=torch.float16, device=device))


def sq_probe_mfma_i8(iters: int, random_operands: bool, fold: bool, sink: torch.Tensor, stream=None,
                     shape: int = 32) -> None:
    """Matrix-core rate probe (include/sq.h): iters * 2^20 int8 MFMA operations
    per wave of a full-occupancy grid, register operands only, on
    v_mfma_i32_32x32x32_i8 (shape 32) or v_mfma_i32_16x16x64_i8 (shape 16);
    sink is int32 scratch of sq_probe_mfma_i8_sink_bytes() bytes."""
    _check(lib().sq_probe_mfma_i8(shape, iters, int(random_operands), int(fold), _ptr(sink), sink.numel() * 4,
                                  _stream(stream)), "sq_probe_mfma_i8")


def sq_probe_mfma_f8f6(fmt: int, iters: int, random_operands: bool, fold: bool, sink: torch.Tensor,
                       stream=None) -> None:
    """The 4-bit path's fp8 / fp6 matrix-core rate probe (include/sq.h): fmt 8
    (e4m3) or 6 (e2m3), iters * 2^20 operations per wave; sink as for
    sq_probe_mfma_i8."""
    _check(lib().sq_probe_mfma_f8f6(fmt, iters, int(random_operands), int(fold), _ptr(sink), sink.numel() * 4,
                                    _stream(stream)), "sq_probe_mfma_f8f6")


def probe_sink(device="cuda") -> torch.Tensor:
    return torch.empty(lib().sq_probe_mfma_i8_sink_bytes() // 4, dtype=torch.int32, device=device)
