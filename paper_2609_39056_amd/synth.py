"""Seeded synthetic inputs shaped like the linears of a world-action DiT.

This module only draws random inputs; it performs none of the quantization
method's arithmetic (no quantizer, no weight folding, no GEMM, no epilogue).
Both the HIP path and the CPU oracle consume what it produces, so it is the one
piece of code they share.

Recipe (what stands in for the paper's Cosmos-Policy / FastWAMJoint /
Cosmos-Edge activations, which are not available):

* Token streams follow the heterogeneous-stream setting of Sec. 3.1: rows are
  grouped into streams (video, proprio, action), stacked contiguously in that
  order (optionally permuted), one stream id per row (the token-wise gain
  diagonal of Fig. 2).
* X: per stream N(0, 1) of shape [n_s, K] times a stream magnitude
  (1, 3, 0.5); a set of outlier input channels (2 % by default, or a per-stream
  fraction) is multiplied by 20; cast to bf16 with round-to-nearest-even.
* W: N(0, 0.02) of shape [N, K] (the transpose of the paper's K x N weight,
  K contiguous), fp32.
* D: a SmoothQuant-style (alpha = 1/2) positive channel scaling
  d_k = clamp(sqrt(amax_k |X| / amax_k |W|), 2^-6, 2^6), computed in fp64 and
  rounded to fp32; dinv_k is the fp32 quotient 1 / d_k.  It stands in for the
  calibrated D* of Sec. 4.2, whose map-weighted objective (Eq. 7) needs a
  trained model.
* bias: N(0, 0.02) as bf16.
* gamma: LogNormal(0, 0.3) of shape [T, S] (a per-step, per-stream gain table,
  Sec. 4.3); clip: per step, the 0.999 quantile of |X D^-1| times
  LogNormal(0, 0.1) (the shared per-step threshold of Sec. 4.3).

The draw order is fixed: outlier channel sets, X per stream, W, bias, gamma,
clip, then the optional row permutation.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

STREAM_NAMES = ("video", "proprio", "action")
STREAM_MAGNITUDE = (1.0, 3.0, 0.5)
OUTLIER_GAIN = 20.0


def _to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns (round-to-nearest-even), via torch's cast."""
    import torch

    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16).copy()


def _bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (b.astype(np.uint32) << 16).view(np.float32)


@dataclass
class LayerInputs:
    """One linear layer's inputs.  Shapes: M rows (tokens), K in, N out."""

    x_bits: np.ndarray          # uint16 [M, K]   bf16 activations
    tok2stream: np.ndarray      # int32  [M]      stream id of each row
    w: np.ndarray               # fp32   [N, K]   full-precision weight (W^T)
    d: np.ndarray               # fp32   [K]      channel scaling D (diagonal)
    dinv: np.ndarray            # fp32   [K]      D^-1
    bias_bits: np.ndarray       # uint16 [N]      bf16 bias
    gamma: np.ndarray           # fp32   [T, S]   per-step per-stream gains
    clip: np.ndarray            # fp32   [T]      per-step shared threshold
    stream_counts: tuple = field(default=())

    @property
    def M(self) -> int:
        return int(self.x_bits.shape[0])

    @property
    def K(self) -> int:
        return int(self.x_bits.shape[1])

    @property
    def N(self) -> int:
        return int(self.w.shape[0])

    @property
    def T(self) -> int:
        return int(self.gamma.shape[0])

    @property
    def S(self) -> int:
        return int(self.gamma.shape[1])


def make_layer(
    K: int,
    N: int,
    stream_counts=(64, 8, 16),
    T: int = 2,
    seed=0,
    outlier_frac=0.02,
    batch: int = 1,
    permute: bool = False,
) -> LayerInputs:
    """Draw one layer's synthetic inputs.

    ``stream_counts`` are the per-sample token counts of (video, proprio,
    action); ``batch`` repeats that three-stream layout per sample.
    ``outlier_frac`` is either one fraction with a single shared channel set
    or a 3-tuple of per-stream fractions with independent channel sets.
    ``seed`` is an int or a sequence of ints (fed to numpy's SeedSequence).
    """
    rng = np.random.default_rng(np.random.SeedSequence(seed))
    S = len(stream_counts)
    per_stream = isinstance(outlier_frac, (tuple, list))
    if per_stream:
        assert len(outlier_frac) == S
        out_sets = [rng.choice(K, size=int(round(f * K)), replace=False) for f in outlier_frac]
    else:
        shared = rng.choice(K, size=int(round(outlier_frac * K)), replace=False)
        out_sets = [shared] * S

    blocks, ids = [], []
    for _ in range(batch):
        for s, n in enumerate(stream_counts):
            if n == 0:
                continue
            xs = rng.standard_normal((n, K)) * STREAM_MAGNITUDE[s % len(STREAM_MAGNITUDE)]
            xs[:, out_sets[s]] *= OUTLIER_GAIN
            blocks.append(xs)
            ids.append(np.full(n, s, dtype=np.int32))
    x64 = np.concatenate(blocks, axis=0)
    tok2stream = np.concatenate(ids)
    x_bits = _to_bf16_bits(x64.astype(np.float32))

    w = (rng.standard_normal((N, K)) * 0.02).astype(np.float32)
    bias_bits = _to_bf16_bits((rng.standard_normal(N) * 0.02).astype(np.float32))
    gamma = rng.lognormal(0.0, 0.3, size=(T, S)).astype(np.float32)

    xf = _bf16_bits_to_f32(x_bits).astype(np.float64)
    amax_x = np.abs(xf).max(axis=0)
    amax_w = np.abs(w.astype(np.float64)).max(axis=0)
    ratio = np.where(amax_w > 0, amax_x / np.where(amax_w > 0, amax_w, 1.0), 1.0)
    d64 = np.clip(np.sqrt(np.where(ratio > 0, ratio, 1.0)), 2.0**-6, 2.0**6)
    d = d64.astype(np.float32)
    dinv = (np.float32(1.0) / d).astype(np.float32)

    q999 = np.quantile(np.abs(xf * dinv.astype(np.float64)), 0.999)
    clip = (q999 * rng.lognormal(0.0, 0.1, size=T)).astype(np.float32)

    if permute:
        perm = rng.permutation(x_bits.shape[0])
        x_bits = np.ascontiguousarray(x_bits[perm])
        tok2stream = np.ascontiguousarray(tok2stream[perm])

    return LayerInputs(
        x_bits=x_bits,
        tok2stream=tok2stream.astype(np.int32),
        w=w,
        d=d,
        dinv=dinv,
        bias_bits=bias_bits,
        gamma=gamma,
        clip=clip,
        stream_counts=tuple(stream_counts),
    )


def device_layer(K: int, N: int, stream_counts=(4096, 32, 64), T: int = 10, seed: int = 0,
                 outlier_frac=0.02, batch: int = 1, device="cuda", with_weight: bool = True) -> dict:
    """The same recipe as make_layer, drawn on the GPU with torch's seeded
    generator, for throughput runs at sizes where drawing on the host is slow.
    Returns device tensors: x (bf16 [M, K]), tok2stream (int32 [M]),
    w (fp32 [N, K], when with_weight), d and dinv (fp32 [K]), bias (bf16 [N]),
    gamma (fp32 [T, S]).  Not bit-identical to make_layer (different
    generator); the parity tests use make_layer."""
    import torch

    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    S = len(stream_counts)
    per_stream = isinstance(outlier_frac, (tuple, list))
    fr = list(outlier_frac) if per_stream else [outlier_frac] * S
    shared = torch.randperm(K, generator=g, device=device)
    sets = [torch.randperm(K, generator=g, device=device)[: int(round(f * K))] if per_stream
            else shared[: int(round(f * K))] for f in fr]
    blocks, ids = [], []
    for _ in range(batch):
        for s, n in enumerate(stream_counts):
            if n == 0:
                continue
            xs = torch.randn((n, K), generator=g, device=device) * STREAM_MAGNITUDE[s % len(STREAM_MAGNITUDE)]
            xs[:, sets[s]] *= OUTLIER_GAIN
            blocks.append(xs)
            ids.append(torch.full((n,), s, dtype=torch.int32, device=device))
    x = torch.cat(blocks).to(torch.bfloat16)
    tok2stream = torch.cat(ids)
    w = torch.randn((N, K), generator=g, device=device) * 0.02
    bias = (torch.randn((N,), generator=g, device=device) * 0.02).to(torch.bfloat16)
    gamma = torch.exp(torch.randn((T, S), generator=g, device=device) * 0.3)
    amax_x = x.float().abs().amax(dim=0).double()
    amax_w = w.abs().amax(dim=0).double()
    ratio = torch.where(amax_w > 0, amax_x / torch.where(amax_w > 0, amax_w, torch.ones_like(amax_w)),
                        torch.ones_like(amax_w))
    d = torch.clamp(torch.sqrt(torch.where(ratio > 0, ratio, torch.ones_like(ratio))), 2.0**-6, 2.0**6).float()
    out = dict(x=x.contiguous(), tok2stream=tok2stream.contiguous(), d=d.contiguous(),
               dinv=(1.0 / d).contiguous(), bias=bias.contiguous(), gamma=gamma.contiguous())
    if with_weight:
        out["w"] = w.contiguous()
    return out


def stratified_rows(tok2stream: np.ndarray, n_video: int = 256, seed: int = 0) -> np.ndarray:
    """Row sample for oracle checks at full size: every row of the small
    streams (id != 0) plus ``n_video`` random rows of stream 0, sorted."""
    rng = np.random.default_rng(seed)
    video = np.flatnonzero(tok2stream == 0)
    other = np.flatnonzero(tok2stream != 0)
    pick = rng.choice(video, size=min(n_video, video.size), replace=False) if video.size else video
    return np.sort(np.concatenate([other, pick])).astype(np.int64)


# The workload configurations (token counts per stream; linears as (K, N)).
SMALL_LAYER = dict(name="single 256x256 linear, 88 tokens", K=256, N=256,
            stream_counts=(64, 8, 16), T=2)
LINEARS_2B = {"qkv": (2048, 6144), "out": (2048, 2048), "up": (2048, 8192), "down": (8192, 2048)}
LINEARS_14B = {"qkv": (5120, 15360), "out": (5120, 5120), "up": (5120, 13824), "down": (13824, 5120)}
TOKENS_2B = (4096, 32, 64)
TOKENS_14B = (8192, 64, 128)
