"""Benchmark of the fused W4A8 / W4A4 linear on one MI355X.

Workload of the headline line: the linears of one 14B-class world-action DiT
block at W4A8 -- qkv 5120->15360, out 5120->5120, up 5120->13824, down
13824->5120 -- over 8384 tokens (8192 video + 64 proprio + 128 action), per-step
per-stream gain tables for 10 denoising steps, int4 weights with fp16 steps per
128-wide group, per-token int8 activations (DYNAMIC range), bf16 output.  This
is the largest layer configuration that runs on one GPU.  One step = one pass
of the hot path over the batch: for each of the four linears, the first kernel
(channel scaling, stream gain, per-token int8 quantization) and the second
(int8-MFMA GEMM against the int4 weight with the dequantization /
compensation / bias epilogue), as one fused C-ABI call per linear
(sq_linear_w4a8).  The denoising step index tau cycles through the table.
Inputs are drawn on the GPU and resident in HBM before the timed region.

A second pass issues the same work as separate sq_quantize_act / sq_gemm_w4a8
calls (the fused call's two launches) with HIP events around every kernel of
every step, on the stream the kernels run on: the per-kernel figures and the
roofline of the GEMM.

Prints one JSON line.  Besides the contract fields it carries the roofline of
the dominant kernel (the GEMM, against the int8 MFMA peak and the matrix-core
rate measured with the same instruction and fold), the fused W4A4 linear, the
unfused variant and the per-output-channel weight steps on the same block, the
2B-class MLP pair (4192 tokens) and the 2B-class block at batch 4 (16768
tokens) as extra records, the MLP chain up -> GELU -> down with and without
the producer-side fusion (14B- and 2B-class shapes), the calibration path (Eq. (9) objective and search,
Eq. (7) scaling objective) on the 2B up projection, and the CPU oracle timed on
a stratified row sample of the 14B block.

Other modes: --suite PATH (every layer configuration and the denoising-loop
sweeps, one JSON record per line) and --action-only TOKENS (the few-token,
weight-streaming regime alone).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_INT8_TOPS = 5000.0      # MI355X dense int8 MFMA, 5.0 POP/s
PEAK_HBM_GBS = 8000.0        # MI355X HBM3E, 8 TB/s
COPY_MIB = 512               # plain device copy run after the timed region (counter calibration)
TRAFFIC_SUMMARY = os.path.join(ROOT, "profiles", "gemm_w4a8_14B_block_M8384_hbm_traffic.md")
GEMM_SOURCES = ("paper_2609_39056_amd/csrc/gemm_w4.hip", "paper_2609_39056_amd/csrc/gemm_frag.h",
                "paper_2609_39056_amd/csrc/sq_internal.h")
T_STEPS = 10
W_GROUP = 128
MLP_2B = (("up", 2048, 8192), ("down", 8192, 2048))


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=100)
    p.add_argument("--warmup", type=int, default=10)
    p.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    p.add_argument("--suite", metavar="PATH", default=None,
                   help="instead of the one-line benchmark, measure every layer configuration (per-layer "
                        "kernels, the unfused path, and the 28-layer x 10-step sweep as one HIP graph) and "
                        "write one JSON record per line to PATH")
    p.add_argument("--action-only", type=int, default=0, metavar="TOKENS",
                   help="time the 2B-class linears on TOKENS action tokens only (the weight-streaming regime): "
                        "28 layers x {qkv, out, up, down} with distinct weights, W4A8 and W4A4, eager calls; "
                        "one JSON line per width (for HBM-traffic counters)")
    p.add_argument("--headline-only", action="store_true",
                   help="only the headline line's own measurements (the 14B block's timed steps, the per-kernel "
                        "pass and the copy that calibrates the byte counters): for kernel traces and counters")
    p.add_argument("--suite-summary", metavar="JSONL",
                   help="print the markdown summary of a --suite run's records (no GPU needed)")
    p.add_argument("--cpu-video-rows", type=int, default=640,
                   help="video rows per layer in the oracle's stratified sample (all proprio / action rows too)")
    return p.parse_args()


def device_block(torch, B, synth, dev, linears, tokens, seed, batch=1, per_channel=False):
    """The linears of one block, drawn on the GPU (synth.device_layer), with
    weights prepared on the GPU (sq_pack_weights).  Keeps each fp32 weight on
    the host for the oracle's baseline leg."""
    layers = []
    for li, (name, (K, N)) in enumerate(linears.items()):
        L = synth.device_layer(K, N, tokens, T=T_STEPS, seed=seed + li, batch=batch, device=dev)
        w = L.pop("w")
        ly = dict(name=name, K=K, N=N, M=int(L["x"].shape[0]), x=L["x"], dev=L,
                  W=B.prepare_weight(w, L["d"], W_GROUP, bias=L["bias"]))
        if per_channel:
            ly["W_pc"] = B.prepare_weight(w, L["d"], K, bias=L["bias"])
        ly["w_host"] = w.cpu().numpy()
        del w
        ly["acts"] = {bits: B.ActParams(tok2stream=L["tok2stream"], gamma=L["gamma"], step=0, act_bits=bits,
                                        dinv=L["dinv"]) for bits in (8, 4)}
        layers.append(ly)
    return layers


def host_layers(torch, B, synth, dev):
    """The 2B-class MLP pair drawn on the host (synth.make_layer), for the
    calibration figures, which need the host inputs."""
    layers = []
    for li, (name, K, N) in enumerate(MLP_2B):
        L = synth.make_layer(K=K, N=N, stream_counts=synth.TOKENS_2B, T=T_STEPS, seed=[0, 2, li])
        x = torch.from_numpy(L.x_bits.view(np.int16)).view(torch.bfloat16).to(dev)
        w, d = torch.from_numpy(L.w).to(dev), torch.from_numpy(L.d).to(dev)
        bias = torch.from_numpy(L.bias_bits.view(np.int16)).view(torch.bfloat16).to(dev)
        W = B.prepare_weight(w, d, W_GROUP, bias=bias)
        W_pc = B.prepare_weight(w, d, K, bias=bias)
        del w
        acts = {bits: B.ActParams(tok2stream=torch.from_numpy(L.tok2stream).to(dev),
                                  gamma=torch.from_numpy(L.gamma).to(dev), step=0, act_bits=bits,
                                  dinv=torch.from_numpy(L.dinv).to(dev)) for bits in (8, 4)}
        layers.append(dict(name=name, K=K, N=N, M=L.M, L=L, x=x, W=W, W_pc=W_pc, acts=acts))
    return layers


def gemm_source_sha256():
    h = hashlib.sha256()
    for rel in GEMM_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def measured_traffic():
    """HBM bytes of one step's four GEMM calls from the committed counter
    summary, or None when there is none or it was taken on a different GEMM
    source."""
    try:
        with open(TRAFFIC_SUMMARY) as f:
            text = f.read()
    except OSError:
        return None
    sha = re.search(r"^source_sha256:\s*([0-9a-f]{64})\s*$", text, re.M)
    val = re.search(r"^traffic_bytes_per_step:\s*([0-9]+)\s*$", text, re.M)
    if not sha or not val or sha.group(1) != gemm_source_sha256():
        return None
    return int(val.group(1))


def cpu_baseline(layers, video_rows):
    """The oracle, as it stands, on a stratified row sample of each linear of
    the block (every proprio and action row plus `video_rows` random video
    rows; each row costs the same arithmetic as in the full layer), W4A8 at
    tau = 3; throughput scaled to TOPS (2 * rows * K * N per second)."""
    import torch

    from oracle import sq_oracle as O
    from paper_2609_39056_amd import synth

    prepared = []
    for ly in layers:  # offline weight preparation and the host copy of the sample: not timed
        d = ly["dev"]
        t2s = d["tok2stream"].cpu().numpy()
        rows = synth.stratified_rows(t2s, video_rows, seed=0)
        xr = ly["x"][torch.as_tensor(rows, device=ly["x"].device)].view(torch.int16).cpu().numpy().view(np.uint16)
        prepared.append(dict(x=xr, t2s=t2s[rows], gamma=d["gamma"].cpu().numpy(), dinv=d["dinv"].cpu().numpy(),
                             bias=d["bias"].view(torch.int16).cpu().numpy().view(np.uint16),
                             pw=O.pack_weights(ly["w_host"], d["d"].cpu().numpy(), W_GROUP), K=ly["K"], N=ly["N"],
                             M=ly["M"]))
    ops = 0
    t0 = time.perf_counter()
    for p in prepared:
        O.linear(p["x"], p["t2s"], p["gamma"], 3, p["pw"]["codes"], p["pw"]["w_scale"], W_GROUP, dinv=p["dinv"],
                 bias_bits=p["bias"], act_bits=8)
        ops += 2 * p["x"].shape[0] * p["K"] * p["N"]
    dt = time.perf_counter() - t0
    try:
        cores = len(os.sched_getaffinity(0))
    except AttributeError:
        cores = os.cpu_count()
    threads = int(os.environ.get("OMP_NUM_THREADS", cores))
    n = prepared[0]["x"].shape[0]
    return dict(value=ops / dt / 1e12, unit="TOPS", cores=min(cores, threads), kind="oracle",
                seconds=round(dt, 3),
                sample=f"stratified rows: {n} of {prepared[0]['M']} per linear (every proprio and action row plus "
                       f"{video_rows} random video rows) of each of the four 14B-block linears (qkv, out, up, "
                       f"down), W4A8 DYNAMIC at tau=3 (quantize, exact block accumulation, fp32 epilogue); "
                       f"weights packed beforehand; throughput extrapolated linearly in rows: "
                       f"TOPS = sum 2*rows*K*N / time")


def suite_summary(path):
    """Markdown tables of a --suite run: per layer, and the denoising sweeps."""
    recs = [json.loads(line) for line in open(path) if line.strip()]
    out = ["# Fused linear, every layer configuration and the denoising sweeps (W4A8 / W4A4)", "",
           "Commands (repo root, one MI355X, ROCm 7.2):", "", "```",
           "python3 bench.py --suite gpurun_out/suite/suite.jsonl",
           "python3 bench.py --suite-summary gpurun_out/suite/suite.jsonl", "```", "",
           "Per-layer times are HIP-event times of one replay of a HIP graph of back-to-back calls (400 for the "
           "256x256 layer, 60 for the 2B layers and the action-only ones, 12 for the 14B layers; a quarter of that for "
           "the unfused path), divided by the call count: device time including each launch's dispatch, not the "
           "host's launch rate; the layer's weight is the same in every call (the denoising sweeps below stream "
           "distinct weights).  K1 = `sq_quantize_act`, K2 = `sq_gemm_w4a*` (main kernel + split tail when there is "
           "one), layer = the fused C-ABI call (K1 + K2), unfused = `sq_linear_unfused`.  With 4-bit activations and "
           "more than 128 tokens the fused call runs its GEMM on the fp8 matrix cores (`gemm_a4f8_kernel`, first "
           "kernel writing fp8 code bytes), while K2 is the stand-alone int8-path GEMM on packed codes.  Fractions: "
           "int8-MFMA peak 5.0 POP/s, HBM 8 TB/s on the algorithmic bytes (bf16 X, int4 W, fp16 steps, bf16 Y, bias, "
           "stream map).  CPU oracle = `oracle/sq_oracle.py` (`linear`, DYNAMIC, the layer's bit width) timed in the "
           "same run on the host's cores: on every row of the small and action-only layers, else on every proprio "
           "and action row plus 64 video rows with the time scaled to all rows (marked *).  Inputs are the seeded "
           "synthetic layers of `synth.device_layer`.", ""]
    for r in recs:
        if r.get("group") == "dispatch cost":
            out += [f"Dispatch cost of one HIP graph node (one-element kernel): **{r['us_per_node']} us**.", ""]
    out += ["| layer | act | weight steps | M | K -> N | K1 us | K2 us | layer us | layer TOPS | K2 % int8 | "
            "layer % HBM | unfused us | fused speedup | CPU oracle us | oracle TOPS | layer / oracle |",
            "|---|---|---|---|---|---|---|---|---|---|---|---|---|---|---|---|"]
    for r in recs:
        if "linear" not in r:
            continue
        steps = "per channel" if r["w_group"] == r["K"] else f"groups of {r['w_group']}"
        orc = ("—", "—", "—")
        if "cpu_oracle_us" in r:
            star = "*" if r["cpu_oracle_extrapolated"] else ""
            orc = (f"{r['cpu_oracle_us']:.0f}{star}", f"{r['cpu_oracle_tops']:.4f}",
                   f"{r['cpu_oracle_us'] / r['us_layer']:.0f}x")
        out.append(f"| {r['group']} {r['linear']} | A{r['act_bits']} | {steps} | {r['M']} | {r['K']} -> {r['N']} | "
                   f"{r['us_quant']:.2f} | {r['us_gemm']:.2f} | {r['us_layer']:.2f} | {r['tops_layer']:.1f} | "
                   f"{100 * r['frac_int8_gemm']:.1f} | {100 * r['frac_hbm_layer']:.2f} | {r['us_unfused']:.2f} | "
                   f"{r['fused_speedup']:.2f} | {orc[0]} | {orc[1]} | {orc[2]} |")
    cores = {r["cpu_cores"] for r in recs if "cpu_cores" in r}
    if cores:
        out += ["", f"CPU oracle threads: {', '.join(str(c) for c in sorted(cores))}."]
    out += ["", "Denoising sweep: 28 layers x 10 steps x {qkv, out, up, down} of the 2B class, each layer with its own "
            "weights (0.7 GB packed, more than the 256 MB MALL), 1120 fused calls captured as one HIP graph:", "",
            "| variant | act | graph ms | eager ms | us per call | TOPS | % int8 | GB/s | % HBM |",
            "|---|---|---|---|---|---|---|---|---|"]
    for r in recs:
        if "variant" in r:
            out.append(f"| {r['variant']} | A{r['act_bits']} | {r['ms_graph']:.2f} | {r['ms_eager']:.2f} | "
                       f"{r['us_per_call']:.2f} | {r['tops']:.1f} | {100 * r['frac_int8']:.2f} | {r['gbs']:.0f} | "
                       f"{100 * r['frac_hbm']:.2f} |")
    print("\n".join(out))


def run_suite(args):
    """Every layer configuration, one JSON record per measurement."""
    import torch

    from paper_2609_39056_amd import binding as B
    from paper_2609_39056_amd import synth

    dev = "cuda:0"
    torch.cuda.set_device(0)
    B.lib()
    BF16 = B.SQ_OUT_BF16
    fout = open(args.suite, "w")

    def emit(rec):
        line = json.dumps(rec)
        print(line, flush=True)
        fout.write(line + "\n")
        fout.flush()

    def timed(fn, reps, warm=3, graph=True):
        """Device time per call: `reps` calls captured as one HIP graph, so the
        host's launch rate does not bound small layers; one warm replay, then
        one timed replay.  graph=False times `reps` eager calls (for fn that
        replays a graph itself)."""
        for _ in range(warm):
            fn()
        torch.cuda.synchronize()
        if not graph:
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(reps):
                fn()
            e1.record()
            torch.cuda.synchronize()
            return e0.elapsed_time(e1) * 1e3 / reps
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for _ in range(reps):
                fn()
        g.replay()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        g.replay()
        e1.record()
        torch.cuda.synchronize()
        del g
        return e0.elapsed_time(e1) * 1e3 / reps  # us per call

    def alg_bytes(M, K, N, wg=W_GROUP):  # bf16 X, int4 W, fp16 steps, bf16 Y, bias, stream map
        return M * K * 2 + N * K // 2 + (K // wg) * N * 2 + M * N * 2 + 2 * N + 4 * M

    def oracle_record(L, w_host, G, bits, step):
        """The oracle, as it stands, on the layer's stratified rows (every
        proprio and action row plus SUITE_ORACLE_VIDEO_ROWS video rows: all
        rows of the small and action-only layers), W4A8 / W4A4 DYNAMIC; time
        extrapolated linearly to all M rows when sampled.  The weight packing
        (offline) is not timed."""
        from oracle import sq_oracle as O
        M, K = L["x"].shape
        N = w_host.shape[0]
        t2s = L["tok2stream"].cpu().numpy()
        rows = synth.stratified_rows(t2s, SUITE_ORACLE_VIDEO_ROWS, seed=0)
        xr = L["x"][torch.as_tensor(rows, device=dev)].view(torch.int16).cpu().numpy().view(np.uint16)
        pw = O.pack_weights(w_host, L["d"].cpu().numpy(), G)
        gamma, dinv = L["gamma"].cpu().numpy(), L["dinv"].cpu().numpy()
        bias = L["bias"].view(torch.int16).cpu().numpy().view(np.uint16)
        t0 = time.perf_counter()
        O.linear(xr, t2s[rows], gamma, step, pw["codes"], pw["w_scale"], G, dinv=dinv, bias_bits=bias,
                 act_bits=bits)
        dt = time.perf_counter() - t0
        us = dt * 1e6 * M / len(rows)
        try:
            cores = len(os.sched_getaffinity(0))
        except AttributeError:
            cores = os.cpu_count()
        return dict(cpu_oracle_us=round(us, 1), cpu_oracle_tops=round(2.0 * M * K * N / us / 1e6, 5),
                    cpu_oracle_rows=int(len(rows)), cpu_oracle_extrapolated=bool(len(rows) < M),
                    cpu_cores=min(cores, int(os.environ.get("OMP_NUM_THREADS", cores))))

    def layer_record(group, name, L, W, bits, reps, w_host=None):
        M, K = L["x"].shape
        N = W.N
        act = B.ActParams(tok2stream=L["tok2stream"], gamma=L["gamma"], step=min(3, L["gamma"].shape[0] - 1),
                          act_bits=bits, dinv=L["dinv"])
        qx, sc = B.act_buffers(M, K, bits, dev)
        wsg = B.alloc_workspace(B.SQ_VARIANT_GEMM, M, K, N, bits, dev)
        wsf = B.alloc_workspace(B.SQ_VARIANT_FUSED, M, K, N, bits, dev)
        wsu = B.alloc_workspace(B.SQ_VARIANT_UNFUSED, M, K, N, bits, dev)
        y = torch.empty((M, N), dtype=torch.bfloat16, device=dev)
        us_k1 = timed(lambda: B.sq_quantize_act(L["x"], act, qx, sc), reps)
        if bits == 8:
            us_k2 = timed(lambda: B.sq_gemm_w4a8(qx, sc, W, y, BF16, workspace=wsg), reps)
        else:
            us_k2 = timed(lambda: B.sq_gemm_w4a4(qx, sc, act, W, y, BF16, workspace=wsg), reps)
        fused = B.sq_linear_w4a8 if bits == 8 else B.sq_linear_w4a4
        us_api = timed(lambda: fused(L["x"], act, W, y, BF16, wsf), reps)
        us_unf = timed(lambda: B.sq_linear_unfused(L["x"], act, W, y, BF16, wsu), max(3, reps // 4))
        ops = 2.0 * M * K * N
        ab = alg_bytes(M, K, N, W.w_group)
        k1b = M * K * 2 + (M * K if bits == 8 else M * K // 2) + (4 * M if bits == 8 else 2 * M * (K // 64)) + 4 * M
        emit(dict(group=group, linear=name, act_bits=bits, M=M, K=K, N=N, w_group=W.w_group,
                  bound="mfma" if ops / ab >= PEAK_INT8_TOPS / PEAK_HBM_GBS * 1e3 else "hbm",
                  us_quant=round(us_k1, 2), us_gemm=round(us_k2, 2), us_layer=round(us_api, 2),
                  tops_layer=round(ops / us_api / 1e6, 1), tops_gemm=round(ops / us_k2 / 1e6, 1),
                  frac_int8_layer=round(ops / us_api / 1e6 / PEAK_INT8_TOPS, 4),
                  frac_int8_gemm=round(ops / us_k2 / 1e6 / PEAK_INT8_TOPS, 4),
                  gbs_layer=round(ab / us_api / 1e3, 1), frac_hbm_layer=round(ab / us_api / 1e3 / PEAK_HBM_GBS, 4),
                  quant_gbs=round(k1b / us_k1 / 1e3, 1), us_unfused=round(us_unf, 2),
                  fused_speedup=round(us_unf / us_api, 3),
                  **(oracle_record(L, w_host, W.w_group, bits, act.step) if w_host is not None else {})))
        del qx, sc, wsg, wsf, wsu, y

    def layer_group(group, linears, tokens, bits_list, outl, reps, T=10, batch=1, per_channel=False):
        for li, (name, (K, N)) in enumerate(linears.items()):
            L = synth.device_layer(K, N, tokens, T=T, seed=1000 + li, outlier_frac=outl, batch=batch, device=dev)
            w = L.pop("w")
            w_host = None if args.no_cpu else w.cpu().numpy()
            W = B.prepare_weight(w, L["d"], K if per_channel else W_GROUP, bias=L["bias"])
            del w
            for bits in bits_list:
                layer_record(group, name, L, W, bits, reps, w_host)
            del L, W
            torch.cuda.empty_cache()

    # dispatch cost of one HIP graph node: a graph of 150 one-element kernels
    one = torch.zeros(1, device=dev)
    one.add_(1)
    torch.cuda.synchronize()
    gph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(gph):
        for _ in range(150):
            one.add_(1)
    emit(dict(group="dispatch cost", what="one-element kernel per HIP graph node",
              us_per_node=round(timed(gph.replay, 10, warm=2, graph=False) / 150, 2)))
    del gph

    layer_group("single 256x256 linear, 88 tokens (64+8+16), 2 steps", {"small": (256, 256)}, (64, 8, 16),
                (8, 4), 0.02, 400, T=2)
    layer_group("2B-class linears, W4A8, 4192 tokens (4096+32+64)", synth.LINEARS_2B, synth.TOKENS_2B, (8,), 0.02, 60)
    layer_group("2B-class linears, W4A4, 4192 tokens, stream outliers 1%/2%/5%", synth.LINEARS_2B, synth.TOKENS_2B,
                (4,), (0.01, 0.02, 0.05), 60)
    layer_group("14B-class linears, 8384 tokens (8192+64+128)", synth.LINEARS_14B, synth.TOKENS_14B, (8, 4), 0.02, 12)
    layer_group("2B-class linears, W4A8, one weight step per output channel (the paper's weight format)",
                synth.LINEARS_2B, synth.TOKENS_2B, (8,), 0.02, 60, per_channel=True)
    layer_group("14B-class column shards at 8-way tensor parallelism (one GPU's share: N / 8)",
                {"qkv/8": (5120, 1920), "up/8": (5120, 1728)}, synth.TOKENS_14B, (8, 4), 0.02, 24)
    layer_group("14B-class linears, W4A8, one weight step per output channel", synth.LINEARS_14B, synth.TOKENS_14B,
                (8,), 0.02, 12, per_channel=True)
    for M in (64, 128):  # the weight-streaming regime, one layer at a time (its weight stays cached across calls)
        layer_group(f"2B-class linears, {M} action tokens only", synth.LINEARS_2B, (0, 0, M), (8, 4), 0.02, 60)

    # ---- denoising-loop sweep: 28 layers x 10 steps x {qkv, out, up, down} of
    # the 2B class, every layer with its own weights (0.7 GB packed: more than
    # the 256 MB last-level cache), captured as one HIP graph
    NL, T = 28, T_STEPS
    lin = synth.LINEARS_2B
    ref = {name: synth.device_layer(K, N, synth.TOKENS_2B, T=T, seed=2000 + i, device=dev, with_weight=False)
           for i, (name, (K, N)) in enumerate(lin.items())}
    g = torch.Generator(device=dev)
    g.manual_seed(7)
    weights = []
    for layer in range(NL):
        ws = {}
        for name, (K, N) in lin.items():
            w = torch.randn((N, K), generator=g, device=dev) * 0.02
            ws[name] = B.prepare_weight(w, ref[name]["d"], W_GROUP, bias=ref[name]["bias"])
            del w
        weights.append(ws)
    torch.cuda.synchronize()
    variants = [("batch 1, 4192 tokens", synth.TOKENS_2B, 1), ("batch 4, 16768 tokens", synth.TOKENS_2B, 4),
                ("action only, 64 tokens", (0, 0, 64), 1), ("action only, 128 tokens", (0, 0, 128), 1)]
    for label, tokens, batch in variants:
        inputs = {name: synth.device_layer(K, N, tokens, T=T, seed=3000 + i, batch=batch, device=dev,
                                           with_weight=False)
                  for i, (name, (K, N)) in enumerate(lin.items())}
        for bits in (8, 4):
            fused = B.sq_linear_w4a8 if bits == 8 else B.sq_linear_w4a4
            bufs = {}
            for name, (K, N) in lin.items():
                M = inputs[name]["x"].shape[0]
                bufs[name] = dict(y=torch.empty((M, N), dtype=torch.bfloat16, device=dev),
                                  ws=B.alloc_workspace(B.SQ_VARIANT_FUSED, M, K, N, bits, dev),
                                  acts=[B.ActParams(tok2stream=inputs[name]["tok2stream"], gamma=inputs[name]["gamma"],
                                                    step=t, act_bits=bits, dinv=inputs[name]["dinv"])
                                        for t in range(T)])

            def sweep_once():
                for t in range(T):
                    for layer in range(NL):
                        for name in lin:
                            b = bufs[name]
                            fused(inputs[name]["x"], b["acts"][t], weights[layer][name], b["y"], BF16, b["ws"])

            sweep_once()  # eager warm-up
            torch.cuda.synchronize()
            us_eager = timed(sweep_once, 2, warm=0, graph=False)
            graph = torch.cuda.CUDAGraph()
            with torch.cuda.graph(graph):
                sweep_once()
            us_graph = timed(graph.replay, 5, warm=2, graph=False)
            calls = T * NL * len(lin)
            ops = T * NL * sum(2.0 * inputs[n]["x"].shape[0] * K * N for n, (K, N) in lin.items())
            ab = T * NL * sum(alg_bytes(inputs[n]["x"].shape[0], K, N) for n, (K, N) in lin.items())
            emit(dict(group="denoising sweep: 28 layers x 10 steps x {qkv, out, up, down}, 2B class, one HIP graph",
                      variant=label, act_bits=bits, calls=calls, tokens=int(inputs["up"]["x"].shape[0]),
                      ms_graph=round(us_graph / 1e3, 3), ms_eager=round(us_eager / 1e3, 3),
                      us_per_call=round(us_graph / calls, 2), tops=round(ops / us_graph / 1e6, 1),
                      frac_int8=round(ops / us_graph / 1e6 / PEAK_INT8_TOPS, 4),
                      gbs=round(ab / us_graph / 1e3, 1), frac_hbm=round(ab / us_graph / 1e3 / PEAK_HBM_GBS, 4)))
            del graph, bufs
        del inputs
        torch.cuda.empty_cache()
    fout.close()


SUITE_ORACLE_VIDEO_ROWS = 64  # video rows per layer in the suite's oracle timing (plus every other row)
PEAK_FP64_TFLOPS = 78.6     # MI355X fp64 (vector and matrix), 78.6 TFLOP/s
CALIB_CANDIDATES = 16
CALIB_ROUNDS = 8


def calibration_figures(torch, B, ly, stream, dev, cpu_rows):
    """The calibration path of Eq. (9) on the up projection (2048 -> 8192,
    one weight step per output channel as in the paper's calibration setup)
    over one batch of M tokens: the fp64 target X~ W^ (once per linear), the
    objective of a batch of candidates (each: the fused linear in STATIC mode,
    fp32 out, then the weighted squared error), the fused linear alone on the
    same tables, the constrained search, and the shared-scaling objective of
    Eq. (7) over 11 exponents of the D family.  HIP events on the stream the
    kernels run on."""
    L, W = ly["L"], ly["W_pc"]
    M, K, N = L.M, ly["K"], ly["N"]
    S = L.gamma.shape[1]
    x, t2s, dinv = ly["x"], ly["acts"][8].tok2stream, ly["acts"][8].dinv
    rng = np.random.default_rng(7)
    gam = (L.gamma[rng.integers(0, L.gamma.shape[0], CALIB_CANDIDATES)]
           * rng.lognormal(0.0, 0.2, (CALIB_CANDIDATES, S))).astype(np.float32)
    clip = (L.clip[0] * rng.lognormal(0.0, 0.3, CALIB_CANDIDATES)).astype(np.float32)
    gam_d, clip_d = torch.from_numpy(gam).to(dev), torch.from_numpy(clip).to(dev)
    omega = torch.full((S,), 1.0 / S, dtype=torch.float64, device=dev)
    ref = torch.empty((M, N), dtype=torch.float64, device=dev)
    obj = torch.empty((CALIB_CANDIDATES,), dtype=torch.float64, device=dev)
    ws = torch.empty(B.sq_calib_search_workspace_bytes(M, K, N, 8, S), dtype=torch.uint8, device=dev)

    def timed(fn, reps):
        fn()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps  # ms

    ms_ref = timed(lambda: B.sq_calib_reference(x, dinv, W, ref, stream), 3)
    ms_obj = timed(lambda: B.sq_calib_objective(x, t2s, S, dinv, 8, W, ref, gam_d, clip_d, omega, obj, ws, stream),
                   3) / CALIB_CANDIDATES
    y32 = torch.empty((M, N), dtype=torch.float32, device=dev)
    wsf = B.alloc_workspace(B.SQ_VARIANT_FUSED, M, K, N, 8, dev)
    Wnb = B.Weight(qw=W.qw, w_scale=W.w_scale, w_group=W.w_group, bias=None)
    act1 = B.ActParams(tok2stream=t2s, gamma=gam_d[:1], step=0, act_bits=8, range_mode=B.SQ_RANGE_STATIC,
                       clip=clip_d[:1], dinv=dinv)
    ms_lin = timed(lambda: B.sq_linear_w4a8(x, act1, Wnb, y32, B.SQ_OUT_F32, wsf, stream), 3 * CALIB_CANDIDATES)
    del y32, wsf
    params = B.sq_calib_search_params(0.25, 4.0, float(L.clip[0]) / 8, float(L.clip[0]) * 4, float(L.clip[0]), 0.5,
                                      CALIB_ROUNDS)
    g_out = torch.empty((S,), dtype=torch.float32, device=dev)
    c_out = torch.empty((1,), dtype=torch.float32, device=dev)
    o_out = torch.empty((1,), dtype=torch.float64, device=dev)
    ms_search = timed(lambda: B.sq_calib_search(x, t2s, S, dinv, 8, W, ref, omega, params, g_out, c_out, o_out, ws,
                                                stream), 1)
    n_search = 1 + CALIB_ROUNDS * 2 * (S + 1)
    start = obj.new_empty((1,))
    B.sq_calib_objective(x, t2s, S, dinv, 8, W, ref, torch.ones((1, S), dtype=torch.float32, device=dev),
                         torch.tensor([float(L.clip[0])], dtype=torch.float32, device=dev), omega, start, ws, stream)
    torch.cuda.synchronize()
    # the shared scaling of Eq. 7 over 11 exponents: full-precision fp64 target,
    # then per exponent D, Q(D W) packed on the GPU, the fused linear (DYNAMIC,
    # unit gains) and the error weighted per stream (uniform)
    alphas = [i / 10 for i in range(11)]
    w32 = torch.from_numpy(L.w).to(dev)
    ref_fp = torch.empty((M, N), dtype=torch.float64, device=dev)
    ms_fp_ref = timed(lambda: B.sq_calib_fp_reference(x, w32, ref_fp, stream), 1)
    ws_s = torch.empty(B.sq_calib_scaling_workspace_bytes(M, K, N, K, 8, S), dtype=torch.uint8, device=dev)
    obj_s = torch.empty((len(alphas),), dtype=torch.float64, device=dev)
    ms_scaling = timed(lambda: B.sq_calib_scaling_objective(x, t2s, S, omega, w32, K, 8, ref_fp, alphas, obj_s, ws_s,
                                                            stream), 1)
    scal = obj_s.cpu().numpy()
    del ws_s, ref_fp, w32
    err_bytes = M * N * (4 + 8)  # the candidate's fp32 output and the fp64 target, read once
    us_err = (ms_obj - ms_lin) * 1e3
    out = {
        "workload": f"up projection {K}->{N}, per-channel int4 weights, M={M} tokens in {S} streams, A8 STATIC",
        "reference_ms": round(ms_ref, 3),
        "reference_fp64_tflops": round(2.0 * M * K * N / (ms_ref * 1e-3) / 1e12, 2),
        "reference_frac_fp64_peak": round(2.0 * M * K * N / (ms_ref * 1e-3) / 1e12 / PEAK_FP64_TFLOPS, 4),
        "objective_us_per_candidate": round(ms_obj * 1e3, 1),
        "fused_linear_f32_us": round(ms_lin * 1e3, 1),
        "error_kernels_us": round(us_err, 1),
        "error_kernels_gbs": round(err_bytes / max(us_err, 1e-3) / 1e3, 1),
        "search_ms": round(ms_search, 2), "search_rounds": CALIB_ROUNDS, "search_candidates": n_search,
        "search_objective_start": float(start.item()), "search_objective_end": float(o_out.item()),
        "search_gamma": [round(float(v), 5) for v in g_out.cpu()], "search_clip": round(float(c_out.item()), 5),
        "scaling_fp_reference_ms": round(ms_fp_ref, 3),
        "scaling_objective_us_per_exponent": round(ms_scaling * 1e3 / len(alphas), 1),
        "scaling_exponents": len(alphas),
        "scaling_best_alpha": alphas[int(np.argmin(scal))],
        "scaling_objective_best": float(scal.min()), "scaling_objective_alpha0": float(scal[0]),
    }
    if cpu_rows is not None:
        out["cpu_oracle"] = calibration_cpu(L, K, cpu_rows)
        out["cpu_oracle"]["gpu_over_cpu"] = round(
            (M / (ms_obj * 1e-3)) / out["cpu_oracle"]["tokens_per_s_per_candidate"], 1)
    return out


def calibration_cpu(L, K, rows):
    """The oracle's Eq. (9) objective for one candidate on a row sample of
    the same layer (its target X~ W^ included, as the GPU's per-linear
    reference is amortized only over candidates)."""
    from oracle import sq_oracle as O

    idx = np.sort(np.random.default_rng(1).choice(L.M, size=rows, replace=False))
    pw = O.pack_weights(L.w, L.d, K)
    S = L.gamma.shape[1]
    t0 = time.perf_counter()
    O.calib_objective(L.x_bits[idx], L.tok2stream[idx], S, pw["codes"], pw["w_scale"], K, L.gamma[:1], L.clip[:1],
                      np.full(S, 1.0 / S), dinv=L.dinv, act_bits=8)
    dt = time.perf_counter() - t0
    return dict(tokens_per_s_per_candidate=round(rows / dt, 1), seconds=round(dt, 3), rows=rows)


def graph_us(torch, fn, reps, warm=3):
    """Device time per call: `reps` calls captured as one HIP graph, one warm
    replay, then one timed replay (HIP events)."""
    for _ in range(warm):
        fn()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for _ in range(reps):
            fn()
    g.replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    g.replay()
    e1.record()
    torch.cuda.synchronize()
    del g
    return e0.elapsed_time(e1) * 1e3 / reps


def static_single_kernel_figures(torch, B, synth, dev, reps=50):
    """The STATIC single-kernel W4A8 linear (sq_linear_w4a8_static1) against
    the two-kernel fused call in STATIC mode (sq_linear_w4a8), at 64 and 128
    action tokens on the 2B-class linears: us per call, graph-replayed."""
    out = {}
    for M in (64, 128):
        for i, (name, (K, N)) in enumerate(synth.LINEARS_2B.items()):
            L = synth.device_layer(K, N, (0, 0, M), T=T_STEPS, seed=7000 + i, device=dev)
            W = B.prepare_weight(L["w"], L["d"], W_GROUP, bias=L["bias"])
            clip = torch.full((T_STEPS,), 4.0, dtype=torch.float32, device=dev)
            act = B.ActParams(tok2stream=L["tok2stream"], gamma=L["gamma"], step=1, act_bits=8,
                              range_mode=B.SQ_RANGE_STATIC, clip=clip, dinv=L["dinv"])
            y = torch.empty((M, N), dtype=torch.bfloat16, device=dev)
            wsf = B.alloc_workspace(B.SQ_VARIANT_FUSED, M, K, N, 8, dev)
            wsg = B.alloc_workspace(B.SQ_VARIANT_GEMM, M, K, N, 8, dev)
            two = graph_us(torch, lambda: B.sq_linear_w4a8(L["x"], act, W, y, B.SQ_OUT_BF16, wsf), reps)
            one = graph_us(torch, lambda: B.sq_linear_w4a8_static1(L["x"], act, W, y, B.SQ_OUT_BF16, wsg), reps)
            out[f"{name}_M{M}"] = dict(us_two_kernels=round(two, 2), us_single_kernel=round(one, 2),
                                       single_over_two=round(one / two, 3))
            del L, W, y, wsf, wsg
    return out


def hbm_copy_figure(torch, dev, stream):
    """A plain device copy of COPY_MIB MiB (a torch copy kernel): the reference
    for the HBM byte counters (FETCH_SIZE / WRITE_SIZE) of profiled launches."""
    src = torch.empty(COPY_MIB << 20, dtype=torch.uint8, device=dev).fill_(1)
    dst = torch.empty_like(src)
    dst.copy_(src)
    c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    c0.record(stream)
    dst.copy_(src)
    c1.record(stream)
    torch.cuda.synchronize()
    us = c0.elapsed_time(c1) * 1e3
    del src, dst
    return {"bytes": 2 * (COPY_MIB << 20), "us": round(us, 1), "gbs": round(2 * (COPY_MIB << 20) / (us * 1e-6) / 1e9, 1)}


def mlp_chain_figures(torch, B, dev, up, down, reps=20, bits=8):
    """The MLP's direct chain, up projection -> GELU -> down projection, with
    the down projection's STATIC quantizer (its per-step thresholds):
    unfused as three calls (the fused linear to bf16, sq_gelu_bf16, the fused
    linear of the down projection) against the producer-side fusion (the
    linear with the GELU epilogue writing the down projection's codes and
    steps, then the down projection's GEMM on them).  bits 8: W4A8
    (sq_linear_w4a8_gelu_quant, sq_gemm_w4a8); bits 4: W4A4
    (sq_linear_w4a4_gelu_quant, then sq_gemm_w4a4 on packed codes up to 128
    tokens, sq_gemm_w4a4_fp8 on fp8 code bytes above).  us per chain and per
    call, graph-replayed; the same tokens feed both projections."""
    M, N, K2 = up["M"], up["N"], down["N"]
    ua, da = up["acts"][bits], down["acts"][bits]
    ua.step = 1
    clip = torch.full((T_STEPS,), 4.0 if bits == 8 else 3.0, dtype=torch.float32, device=dev)
    dact = B.ActParams(tok2stream=ua.tok2stream, gamma=da.gamma, step=1, act_bits=bits,
                       range_mode=B.SQ_RANGE_STATIC, clip=clip, dinv=da.dinv)
    h = torch.empty((M, N), dtype=torch.bfloat16, device=dev)
    g = torch.empty_like(h)
    yd = torch.empty((M, K2), dtype=torch.bfloat16, device=dev)
    ws_up = B.alloc_workspace(B.SQ_VARIANT_FUSED, M, up["K"], N, bits, dev)
    ws_dn = B.alloc_workspace(B.SQ_VARIANT_FUSED, M, N, K2, bits, dev)
    ws_g = B.alloc_workspace(B.SQ_VARIANT_GEMM, M, N, K2, bits, dev)
    kn = None
    if bits == 8 or M <= 128:
        qn, sn = B.act_buffers(M, N, bits, dev)
    else:
        qn = torch.empty((M, N), dtype=torch.uint8, device=dev)
        sn = torch.empty((M, N // B.A4_GROUP), dtype=torch.float32, device=dev)
        kn = torch.empty_like(sn)
    BF = B.SQ_OUT_BF16
    if bits == 8:
        linear = B.sq_linear_w4a8
        gelu_quant = lambda: B.sq_linear_w4a8_gelu_quant(up["x"], ua, up["W"], dact, qn, sn, ws_up)
        down_gemm = lambda: B.sq_gemm_w4a8(qn, sn, down["W"], yd, BF, workspace=ws_g)
    else:
        linear = B.sq_linear_w4a4
        gelu_quant = lambda: B.sq_linear_w4a4_gelu_quant(up["x"], ua, up["W"], dact, qn, sn, kn, ws_up)
        if kn is None:
            down_gemm = lambda: B.sq_gemm_w4a4(qn, sn, dact, down["W"], yd, BF, workspace=ws_g)
        else:
            down_gemm = lambda: B.sq_gemm_w4a4_fp8(qn, sn, kn, dact, down["W"], yd, BF, workspace=ws_g)
    calls = {
        "up_linear_bf16": lambda: linear(up["x"], ua, up["W"], h, BF, ws_up),
        "gelu_bf16": lambda: B.sq_gelu_bf16(h, g),
        "down_linear_static": lambda: linear(g, dact, down["W"], yd, BF, ws_dn),
        "up_linear_gelu_quant": gelu_quant,
        "down_gemm": down_gemm,
    }
    per = {k: round(graph_us(torch, f, reps), 2) for k, f in calls.items()}

    def unfused():
        for k in ("up_linear_bf16", "gelu_bf16", "down_linear_static"):
            calls[k]()

    def fused():
        for k in ("up_linear_gelu_quant", "down_gemm"):
            calls[k]()

    us_u = graph_us(torch, unfused, reps)
    us_f = graph_us(torch, fused, reps)
    ops = 2.0 * M * up["K"] * N + 2.0 * M * N * K2
    del h, g, yd, ws_up, ws_dn, ws_g, qn, sn, kn
    return {"M": M, "act_bits": bits, "up": [up["K"], N], "down": [N, K2], "per_call_us": per,
            "unfused_us": round(us_u, 2), "fused_us": round(us_f, 2), "fused_speedup": round(us_u / us_f, 3),
            "fused_tops": round(ops / (us_f * 1e-6) / 1e12, 1), "unfused_tops": round(ops / (us_u * 1e-6) / 1e12, 1)}


def run_action_only(args):
    """The few-token regime: every call streams a distinct weight (28 layers x
    4 linears, 0.7 GB packed: more than the 256 MB last-level cache), one pass
    of eager fused calls per width, HIP events around the pass, then a plain
    512 MiB copy (the reference for the HBM byte counters)."""
    import torch

    from paper_2609_39056_amd import binding as B
    from paper_2609_39056_amd import synth

    dev = "cuda:0"
    torch.cuda.set_device(0)
    B.lib()
    stream = torch.cuda.current_stream()
    tokens = (0, 0, args.action_only)
    lin = synth.LINEARS_2B
    NL = 28
    inputs = {name: synth.device_layer(K, N, tokens, T=T_STEPS, seed=4000 + i, device=dev, with_weight=False)
              for i, (name, (K, N)) in enumerate(lin.items())}
    g = torch.Generator(device=dev)
    g.manual_seed(11)
    weights = []
    for _ in range(NL):
        ws = {}
        for name, (K, N) in lin.items():
            w = torch.randn((N, K), generator=g, device=dev) * 0.02
            ws[name] = B.prepare_weight(w, inputs[name]["d"], W_GROUP, bias=inputs[name]["bias"])
            del w
        weights.append(ws)
    M = args.action_only
    for bits in (8, 4):
        fused = B.sq_linear_w4a8 if bits == 8 else B.sq_linear_w4a4
        bufs = {name: dict(y=torch.empty((M, N), dtype=torch.bfloat16, device=dev),
                           ws=B.alloc_workspace(B.SQ_VARIANT_FUSED, M, K, N, bits, dev),
                           act=B.ActParams(tok2stream=inputs[name]["tok2stream"], gamma=inputs[name]["gamma"],
                                           step=1, act_bits=bits, dinv=inputs[name]["dinv"]))
                for name, (K, N) in lin.items()}

        def one_pass():
            for layer in range(NL):
                for name in lin:
                    b = bufs[name]
                    fused(inputs[name]["x"], b["act"], weights[layer][name], b["y"], B.SQ_OUT_BF16, b["ws"], stream)

        for _ in range(max(1, args.warmup // 10)):
            one_pass()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        one_pass()
        e1.record(stream)
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) * 1e3
        calls = NL * len(lin)
        ab = NL * sum(M * K * 2 + N * K // 2 + N * K // W_GROUP * 2 + M * N * 2 + 2 * N + 4 * M
                      for K, N in lin.values())
        print(json.dumps(dict(group="action-only linears, 2B class, eager fused calls", tokens=M, act_bits=bits,
                              calls=calls, us_per_call=round(us / calls, 2), alg_mb_per_pass=round(ab / 1e6, 1),
                              gbs=round(ab / us / 1e3, 1), frac_hbm=round(ab / us / 1e3 / PEAK_HBM_GBS, 4))),
              flush=True)
        del bufs
    src = torch.empty(COPY_MIB << 20, dtype=torch.uint8, device=dev).fill_(1)
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only; --gpus {args.gpus} is not supported (every step of the layer is "
              f"row-independent: several GPUs would each take their own slice of the tokens)", file=sys.stderr)
        sys.exit(2)
    if args.action_only:
        run_action_only(args)
        return
    if args.suite_summary:
        suite_summary(args.suite_summary)
        return
    if args.suite:
        run_suite(args)
        return

    import torch

    from paper_2609_39056_amd import binding as B
    from paper_2609_39056_amd import synth

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    dev = "cuda:0"
    torch.cuda.set_device(0)
    B.lib()
    stream = torch.cuda.current_stream()
    BF16 = B.SQ_OUT_BF16
    FUSED = {8: B.sq_linear_w4a8, 4: B.sq_linear_w4a4}

    def buffers(layers, with_split=False, unfused=False):
        for ly in layers:
            M, K, N = ly["M"], ly["K"], ly["N"]
            ly["y"] = torch.empty((M, N), dtype=torch.bfloat16, device=dev)
            ly["ws_fused"] = {b: B.alloc_workspace(B.SQ_VARIANT_FUSED, M, K, N, b, dev) for b in (8, 4)}
            if with_split:
                ly["qx8"], ly["r8"] = B.act_buffers(M, K, 8, dev)
                ly["ws_gemm"] = B.alloc_workspace(B.SQ_VARIANT_GEMM, M, K, N, 8, dev)
            if unfused:
                ly["ws_unf"] = B.alloc_workspace(B.SQ_VARIANT_UNFUSED, M, K, N, 8, dev)

    def fused_step(layers, tau, bits=8, wkey="W"):
        for ly in layers:
            act = ly["acts"][bits]
            act.step = tau
            FUSED[bits](ly["x"], act, ly[wkey], ly["y"], BF16, ly["ws_fused"][bits], stream)

    def unfused_step(layers, tau):
        for ly in layers:
            act = ly["acts"][8]
            act.step = tau
            B.sq_linear_unfused(ly["x"], act, ly["W"], ly["y"], BF16, ly["ws_unf"], stream)

    def timed_steps(step_fn, steps, warmup):
        """Wall time per step (ms) of `steps` steps after `warmup` untimed ones,
        synchronized on both sides."""
        for s in range(warmup):
            step_fn(s % T_STEPS)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for s in range(steps):
            step_fn(s % T_STEPS)
        torch.cuda.synchronize()
        return (time.perf_counter() - t0) * 1e3 / steps

    def event_pass(layers, calls, steps):
        """Per-call device time: HIP events on the kernels' stream around
        every call of every step; calls(ly, tau) issues one layer's calls in
        order and returns their count.  Returns (ms per call [layer][call],
        wall ms per step)."""
        ncall = None
        evs = []
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for s in range(steps):
            e = []
            for ly in layers:
                e.append(torch.cuda.Event(enable_timing=True))
                e[-1].record(stream)
                n = calls(ly, s % T_STEPS, e)
                ncall = n if ncall is None else ncall
            e.append(torch.cuda.Event(enable_timing=True))
            e[-1].record(stream)
            evs.append(e)
        torch.cuda.synchronize()
        wall = (time.perf_counter() - t0) * 1e3 / steps
        per = np.zeros((len(layers), ncall))
        for e in evs:
            for i in range(len(layers)):
                for c in range(ncall):
                    k = i * ncall + c
                    per[i, c] += e[k].elapsed_time(e[k + 1])
        return per / steps, wall

    def split_calls(ly, tau, e):
        act = ly["acts"][8]
        act.step = tau
        B.sq_quantize_act(ly["x"], act, ly["qx8"], ly["r8"], stream)
        e.append(torch.cuda.Event(enable_timing=True))
        e[-1].record(stream)
        B.sq_gemm_w4a8(ly["qx8"], ly["r8"], ly["W"], ly["y"], BF16, workspace=ly["ws_gemm"], stream=stream)
        return 2

    def fused_calls(bits):
        def calls(ly, tau, e):
            act = ly["acts"][bits]
            act.step = tau
            FUSED[bits](ly["x"], act, ly["W"], ly["y"], BF16, ly["ws_fused"][bits], stream)
            return 1
        return calls

    def ops_of(layers):
        return sum(2.0 * ly["M"] * ly["K"] * ly["N"] for ly in layers)

    # ---- the 14B-class block (configuration 4), drawn on the GPU
    blk = device_block(torch, B, synth, dev, synth.LINEARS_14B, synth.TOKENS_14B, seed=5000, per_channel=True)
    buffers(blk, with_split=True, unfused=True)
    M = blk[0]["M"]
    ops_step = ops_of(blk)

    # ---- headline timed region: the fused W4A8 linear (sq_linear_w4a8, the
    # product's entry point) for the four linears, K steps
    ms_per_step = timed_steps(lambda t: fused_step(blk, t), args.steps, args.warmup)
    value = ops_step / (ms_per_step * 1e-3) / 1e12

    # ---- per-kernel pass: the same steps as the fused call's two launches,
    # events around every kernel of every step
    for s in range(max(2, args.warmup // 2)):
        for ly in blk:
            split_calls(ly, s % T_STEPS, [])
    per_k, ms_split = event_pass(blk, split_calls, args.steps)
    k1, k2 = per_k[:, 0], per_k[:, 1]  # ms per launch, per linear
    ops = [2.0 * M * ly["K"] * ly["N"] for ly in blk]
    gemm_tops = sum(ops) / (k2.sum() * 1e-3) / 1e12
    # algorithmic bytes: first kernel bf16 X in, int8 Q_X + fp32 r out (+ the
    # stream map); GEMM Q_X + r in, int4 W + fp16 steps + bf16 bias, bf16 Y out;
    # layer bf16 X, int4 W, fp16 steps, bias, bf16 Y, stream map
    k1_bytes = [M * ly["K"] * 3 + 8 * M for ly in blk]
    k2_bytes = [M * ly["K"] + 4 * M + ly["N"] * ly["K"] // 2 + ly["N"] * ly["K"] // W_GROUP * 2 + 2 * ly["N"]
                + 2 * M * ly["N"] for ly in blk]
    alg_bytes = [M * ly["K"] * 2 + ly["N"] * ly["K"] // 2 + ly["N"] * ly["K"] // W_GROUP * 2 + 2 * ly["N"]
                 + M * ly["N"] * 2 + 4 * M for ly in blk]
    serial = [b1 / (PEAK_HBM_GBS * 1e9) + max(o / (PEAK_INT8_TOPS * 1e12), b2 / (PEAK_HBM_GBS * 1e9))
              for b1, b2, o in zip(k1_bytes, k2_bytes, ops)]
    per_layer = {}
    for i, ly in enumerate(blk):
        t = (k1[i] + k2[i]) * 1e-3
        per_layer[ly["name"]] = dict(
            K=ly["K"], N=ly["N"], us_quant=round(k1[i] * 1e3, 2), us_gemm=round(k2[i] * 1e3, 2),
            us_layer=round(t * 1e6, 2), tops_layer=round(ops[i] / t / 1e12, 1),
            tops_gemm=round(ops[i] / (k2[i] * 1e-3) / 1e12, 1),
            frac_layer_int8=round(ops[i] / t / 1e12 / PEAK_INT8_TOPS, 4),
            frac_gemm_int8=round(ops[i] / (k2[i] * 1e-3) / 1e12 / PEAK_INT8_TOPS, 4),
            frac_quant_hbm=round(k1_bytes[i] / (k1[i] * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
            frac_serial_roofline=round(serial[i] / t, 4), alg_mb=round(alg_bytes[i] / 1e6, 2))

    if not args.headline_only:
        # ---- fused W4A4 on the same block, with per-linear call times
        ms_w4a4 = timed_steps(lambda t: fused_step(blk, t, bits=4), args.steps, max(2, args.warmup // 2))
        per4, _ = event_pass(blk, fused_calls(4), max(5, args.steps // 4))
        per8, _ = event_pass(blk, fused_calls(8), max(5, args.steps // 4))
        # ---- unfused W4A8 and per-output-channel weight steps on the same block
        ms_unfused = timed_steps(lambda t: unfused_step(blk, t), max(5, args.steps // 4), 2)
        ms_pc = timed_steps(lambda t: fused_step(blk, t, wkey="W_pc"), args.steps, 2)
        for ly in blk:
            del ly["ws_unf"]
        torch.cuda.empty_cache()
        chain14 = mlp_chain_figures(torch, B, dev, blk[2], blk[3])
        chain14_pc = mlp_chain_figures(torch, B, dev, {**blk[2], "W": blk[2]["W_pc"]},
                                       {**blk[3], "W": blk[3]["W_pc"]})
        chain14_a4 = mlp_chain_figures(torch, B, dev, blk[2], blk[3], bits=4)
        for ly in blk:
            del ly["W_pc"], ly["ws_gemm"], ly["qx8"], ly["r8"]
        torch.cuda.empty_cache()

        # ---- the 2B-class MLP pair (configuration 2) and the 2B-class block at
        # batch 4 (configuration 5's batch-4 row count)
        mlp = host_layers(torch, B, synth, dev)
        buffers(mlp)
        ms_mlp8 = timed_steps(lambda t: fused_step(mlp, t), args.steps, args.warmup)
        ms_mlp4 = timed_steps(lambda t: fused_step(mlp, t, bits=4), args.steps, 2)
        chain2 = mlp_chain_figures(torch, B, dev, mlp[0], mlp[1])
        chain2_a4 = mlp_chain_figures(torch, B, dev, mlp[0], mlp[1], bits=4)
        b4 = device_block(torch, B, synth, dev, synth.LINEARS_2B, synth.TOKENS_2B, seed=6000, batch=4)
        buffers(b4)
        ms_b4 = {bits: timed_steps(lambda t, b=bits: fused_step(b4, t, bits=b), max(10, args.steps // 2), 3)
                 for bits in (8, 4)}
        del b4
        torch.cuda.empty_cache()

        # ---- the STATIC single-kernel linear at few tokens, against the two kernels
        single = static_single_kernel_figures(torch, B, synth, dev)
        # ---- the MLP chain at few tokens (the weight-streaming GEMM with the GELU epilogue)
        chain_few = {}
        for tag, lins, Mf in (("2B_M64", synth.LINEARS_2B, 64), ("2B_M128", synth.LINEARS_2B, 128),
                              ("14B_M64", synth.LINEARS_14B, 64)):
            pair = device_block(torch, B, synth, dev, {"up": lins["up"], "down": lins["down"]}, (0, 0, Mf),
                                seed=7100)
            chain_few[tag] = mlp_chain_figures(torch, B, dev, pair[0], pair[1], reps=50)
            chain_few[tag + "_A4"] = mlp_chain_figures(torch, B, dev, pair[0], pair[1], reps=50, bits=4)
            del pair
        torch.cuda.empty_cache()

        # ---- the calibration path of Eq. (9) on the 2B up projection
        calib = calibration_figures(torch, B, mlp[0], stream, dev, None if args.no_cpu else 256)

        # ---- the 4-bit path's matrix-core rate (sq_probe_mfma_f8f6: the fp8 W4A4
        # GEMM's instruction on fp8 and on fp6 operands, with and without its
        # two-fma fold per output and block)
        sink6 = B.probe_sink(dev)
        n_wg6 = sink6.numel() // 256
        f8f6 = {}
        for fmt, fname in ((8, "fp8"), (6, "fp6")):
            for label, fold in (("random_operands", 0), ("random_operands_with_fold", 1)):
                B.sq_probe_mfma_f8f6(fmt, 200, True, fold, sink6, stream)
                q0, q1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                q0.record(stream)
                B.sq_probe_mfma_f8f6(fmt, 10000, True, fold, sink6, stream)
                q1.record(stream)
                torch.cuda.synchronize()
                f8f6[f"{fname}_{label}"] = round(n_wg6 * 4 * 10000 * 2.0 ** 20 / (q0.elapsed_time(q1) * 1e-3) / 1e12, 1)
        del sink6

    # ---- the int8 matrix-core rate this GPU sustains (sq_probe_mfma_i8: back
    # to back MFMAs on register operands at the GEMM's occupancy) in both MFMA
    # forms: zero operands, random operands, and random operands with the
    # 128-wide block fold of the GEMM kernel that issues that form
    sink = B.probe_sink(dev)
    n_wg = sink.numel() // 256
    probe_iters = 20000
    ceiling = {}
    for shape, name in ((16, "16x16x64"), (32, "32x32x32")):
        for label, rnd, fold in (("zero_operands", 0, 0), ("random_operands", 1, 0),
                                 ("random_operands_with_fold", 1, 1)):
            B.sq_probe_mfma_i8(200, rnd, fold, sink, stream, shape=shape)
            p0, p1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            p0.record(stream)
            B.sq_probe_mfma_i8(probe_iters, rnd, fold, sink, stream, shape=shape)
            p1.record(stream)
            torch.cuda.synchronize()
            probe_ops = n_wg * 4 * probe_iters * 2.0 ** 20
            ceiling[f"{name}_{label}"] = round(probe_ops / (p0.elapsed_time(p1) * 1e-3) / 1e12, 1)
    del sink
    ceil_gemm = ceiling["16x16x64_random_operands_with_fold"]

    # ---- a plain device copy of known size: the reference for the HBM byte
    # counters (FETCH_SIZE / WRITE_SIZE) of the profiled GEMM launches
    copy = hbm_copy_figure(torch, dev, stream)

    out = {
        "metric": "fused W4A8/W4A4 linear TOPS + % int8-MFMA (or HBM) roofline per layer",
        "value": round(value, 2),
        "unit": "TOPS",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int8",
        "data": "synthetic",
        "config": {
            "workload": "14B-class WAM DiT block linears, W4A8: qkv 5120->15360, out 5120->5120, "
                        "up 5120->13824, down 13824->5120; M=8384 tokens (8192 video + 64 proprio + 128 action), "
                        "10-step gain tables, int4 weight groups of 128 (fp16 steps), per-token int8 activations "
                        "(DYNAMIC), bf16 out",
            "M": M, "linears": [[ly["name"], ly["K"], ly["N"]] for ly in blk], "act_bits": 8, "w_group": W_GROUP,
        },
        "roofline": {
            "bound": "mfma",
            "kernel": "sq_gemm_w4a8: gemm_pipe16_kernel<0, false> (+ gemm_tail_kernel<8,0,false> where tiles split)",
            "per": "the four GEMM calls of one step (qkv, out, up, down)",
            "launches": int(args.steps * len(blk)),
            "achieved": round(gemm_tops, 1), "peak": PEAK_INT8_TOPS, "unit": "TOPS",
            "frac": round(gemm_tops / PEAK_INT8_TOPS, 4), "traffic": measured_traffic(),
            "ops_per_step": ops_step, "us_gemm_per_step": round(k2.sum() * 1e3, 2),
            "measured_ceiling": ceil_gemm,
            "measured_ceiling_what": "v_mfma_i32_16x16x64_i8 with the biased 128-block fold, random operands",
            "frac_of_measured_ceiling": round(gemm_tops / ceil_gemm, 4),
        },
        "mfma_i8_ceiling_tops": ceiling,
        **({} if args.headline_only else {"mfma_f8f6_ceiling_tops": f8f6}),
        "per_layer": per_layer,
        "quant_kernel_gbs": round(sum(k1_bytes) / (k1.sum() * 1e-3) / 1e9, 1),
        "w4a8_as_k1_k2_calls": {"ms_per_step": round(ms_split, 5),
                                "gemm_tops": round(gemm_tops, 1)},
        "hbm_copy": copy,
    }
    if not args.headline_only:
        mlp_ops = ops_of(mlp)
        b4_ops = sum(2.0 * 4 * sum(synth.TOKENS_2B) * K * N for K, N in synth.LINEARS_2B.values())
        out.update({
            "fused_w4a8_per_call_us": {ly["name"]: round(per8[i, 0] * 1e3, 2) for i, ly in enumerate(blk)},
            "fused_w4a4": {"ms_per_step": round(ms_w4a4, 5), "tops": round(ops_step / (ms_w4a4 * 1e-3) / 1e12, 2),
                           "per_call_us": {ly["name"]: round(per4[i, 0] * 1e3, 2) for i, ly in enumerate(blk)},
                           "frac_int8": round(ops_step / (ms_w4a4 * 1e-3) / 1e12 / PEAK_INT8_TOPS, 4)},
            "unfused_w4a8": {"ms_per_step": round(ms_unfused, 5),
                             "tops": round(ops_step / (ms_unfused * 1e-3) / 1e12, 2),
                             "fused_speedup": round(ms_unfused / ms_per_step, 3)},
            "fused_w4a8_per_channel_steps": {"ms_per_step": round(ms_pc, 5),
                                             "tops": round(ops_step / (ms_pc * 1e-3) / 1e12, 2)},
            "mlp_2B_M4192": {"workload": "2B-class MLP pair up 2048->8192, down 8192->2048, M=4192 (4096+32+64)",
                             "w4a8": {"ms_per_step": round(ms_mlp8, 5),
                                      "tops": round(mlp_ops / (ms_mlp8 * 1e-3) / 1e12, 2)},
                             "w4a4": {"ms_per_step": round(ms_mlp4, 5),
                                      "tops": round(mlp_ops / (ms_mlp4 * 1e-3) / 1e12, 2)}},
            "mlp_chain_gelu_fusion": {"14B_M8384": chain14, "14B_M8384_per_channel_steps": chain14_pc,
                                      "14B_M8384_A4": chain14_a4, "2B_M4192": chain2, "2B_M4192_A4": chain2_a4,
                                      **chain_few},
            "block_2B_batch4_M16768": {"workload": "2B-class block qkv/out/up/down, batch 4: M=16768",
                                       **{f"w4a{b}": {"ms_per_step": round(ms_b4[b], 5),
                                                      "tops": round(b4_ops / (ms_b4[b] * 1e-3) / 1e12, 2)}
                                          for b in (8, 4)}},
            "static_single_kernel_few_tokens": single,
            "calibration": calib,
        })
    if not args.no_cpu:
        out["cpu_baseline"] = cpu_baseline(blk, args.cpu_video_rows)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
