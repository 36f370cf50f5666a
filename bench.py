"""Benchmark of the fused sparse convolution on one MI355X.

Default workload: the VGG-style block (N=32, 224x224, C=K=64 with 3 real input
channels, two chained 3x3 sparse convs at density 0.2 with fused bias + ReLU,
the second with a fused 2x2 max-pool to 112x112), the largest layer
configuration. One step = the whole hot path on one resident batch: layer 1
forms its input's zero border while staging it in LDS and writes layer 2's
zero-bordered input; layer 2 adds the max-pool. The JSON line (rank 0) carries
the block's nonzero GFLOP/s, ms per step, per-layer times (HIP events on the
launch stream inside the timed steps, and the median of 30 runs each after a
512 MiB write that flushes the last-level cache), a roofline record for the
dominant kernel, the CPU oracle's rate on the same block, and a `per_config`
list with the same measurements for the other layer configurations (the tiny,
ResNet, conv+pool and deep narrow layers).

`--workload NAME` times one other layer or block instead (old single-layer
record), for profiling.
"""
from __future__ import annotations

import argparse
import gc
import hashlib
import json
import os
import statistics
import sys
import time
from pathlib import Path

ROOT = Path(__file__).resolve().parent
sys.path.insert(0, str(ROOT))

HBM_PEAK_GBS = 8000.0           # MI355X HBM3E, published
VALU_FP32_FMA_TFLOPS = 78.6     # 256 CU x 64 lanes x 2 FLOP x 2.4 GHz (v_fma_f32; packed FP32 forms not used)
MFMA_FP32_TFLOPS = 157.3        # MI355X dense fp32 matrix peak, published
FP32_VECTOR_PUBLISHED_TFLOPS = 157.3

WORKLOADS = {
    "resnet": "ResNet-style sparse conv: N=32, C=K=64, 56x56, 3x3, stride 1, pad 1, density 0.2, bias+ReLU, fp32",
    "tiny": "tiny sparse conv: N=1, C=K=16, 16x16, 3x3, stride 1, pad 1, density 0.2, bias+ReLU, fp32",
    "conv_pool": "sparse conv + pool: N=32, C=K=128, 28x28 -> 14x14, 3x3, density 0.1, bias+ReLU+2x2 max-pool, fp32",
    "narrow_d0.05": "deep narrow: N=32, C=K=256, 14x14, 3x3, density 0.05 (Beta(2,5) row skew), bias+ReLU, fp32",
    "narrow_d0.2": "deep narrow: N=32, C=K=256, 14x14, 3x3, density 0.2 (Beta(2,5) row skew), bias+ReLU, fp32",
    "narrow_d0.5": "deep narrow: N=32, C=K=256, 14x14, 3x3, density 0.5 (Beta(2,5) row skew), bias+ReLU, fp32",
}
# Chained blocks: several layers per step, fused through zero-bordered outputs.
BLOCKS = {
    "vgg_block": "VGG-style block: N=32, C=3 padded to 64, 224x224, two chained 3x3 convs C=K=64, density 0.2, "
                 "bias+ReLU, the second with 2x2 max-pool; fp32",
    "resnet_block": "ResNet basic block: N=32, C=K=64, 56x56, relu(conv2(relu(conv1(x))) + x), 3x3 convs, "
                    "density 0.2, bias; fp32",
    "resize_block": "Resize-Conv-ReLU-Maxpool: N=32, C=K=128, bilinear resize 42x42 -> 28x28 (pixel centres "
                    "aligned), 3x3 conv density 0.1, bias+ReLU+2x2 max-pool to 14x14; fp32",
}


def resize_source_bytes(planes, Hin, Win, H, W):
    """Bytes of the source a bilinear resize must read: the source rows and
    columns that some output pixel takes a tap from (all of them unless the
    downscale exceeds 2x), once each."""
    def taps(n_in, n_out):
        used = set()
        for o in range(n_out):
            num = max((2 * o + 1) * n_in - n_out, 0)
            i0 = num // (2 * n_out)
            used.update((i0, min(i0 + 1, n_in - 1)))
        return len(used)
    return 4.0 * planes * taps(Hin, H) * taps(Win, W)


def algorithmic(layer, nnz):
    """Nonzero FLOPs and algorithmic HBM bytes of one fused layer (pad excluded):
    FLOPs = 2 * nnz * N * Ho * Wo; bytes = padded input read once + final output
    written once + 8 B per nonzero (offset, value) + rowptr and bias."""
    N, C, H, W, K, R, S = layer.shape
    Hp, Wp = H + 2 * layer.pad, W + 2 * layer.pad
    Ho = (Hp - R) // layer.stride + 1
    Wo = (Wp - S) // layer.stride + 1
    Hq, Wq = (Ho // 2, Wo // 2) if layer.pool else (Ho, Wo)
    flops = 2.0 * nnz * N * Ho * Wo
    fwd_bytes = 4.0 * N * C * Hp * Wp + 4.0 * N * K * Hq * Wq + 8.0 * nnz + 4.0 * (2 * K + 1)
    pad_bytes = 4.0 * N * C * H * W + 4.0 * N * C * Hp * Wp
    return flops, fwd_bytes, pad_bytes


# Sources of each kernel family: their hash keys the committed counter summaries
# (profiles/spconv_<family>_<workload>_traffic.json).
KERNEL_SOURCES = {
    "fwd": [ROOT / "paper_2005_04091_amd" / "csrc" / f for f in ("spconv.hip", "common.h")],
    "dense": [ROOT / "paper_2005_04091_amd" / "csrc" / f for f in ("dense.hip", "common.h")],
}


def kernel_source_sha(family: str = "fwd") -> str:
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[family]:
        h.update(f.read_bytes())
    return h.hexdigest()[:16]


def measured_traffic(workload: str, family: str = "fwd"):
    """HBM bytes per launch of the forward kernel, from the committed counter
    summary for this workload, or None when it is missing or was taken on a
    different kernel source."""
    f = ROOT / "profiles" / f"spconv_{family}_{workload}_traffic.json"
    if not f.exists():
        return None
    rec = json.loads(f.read_text())
    if rec.get("kernel_source_sha") != kernel_source_sha(family):
        return None
    return rec.get("traffic_bytes")


def copy_calibration(mb: int, dev):
    """A plain device-to-device copy of known size, run three times, so that a
    counter run over this process also records what FETCH_SIZE / WRITE_SIZE read
    for exactly `mb` MiB moved."""
    import torch
    n = mb * 1024 * 1024 // 4
    src = torch.ones(n, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()


def cold_median_ms(fn, stream, reps: int, dev) -> float:
    """Median duration of `fn` with the last-level cache flushed before each
    run: a 512 MiB buffer is written first (the 256 MB MALL cannot hold the
    layer's input from the previous run), then a HIP event pair on the launch
    stream brackets `fn` alone."""
    import torch
    flush = torch.empty(512 * 1024 * 1024 // 4, dtype=torch.float32, device=dev)
    times = []
    for i in range(reps):
        flush.fill_(float(i))
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        fn()
        e1.record(stream)
        torch.cuda.synchronize()
        times.append(e0.elapsed_time(e1))
    del flush
    return statistics.median(times)


def measured_copy_gbs(dev) -> float:
    """Device-to-device copy rate of a 512 MiB tensor through the library's
    pad kernel with pad 0 (a 16-byte-per-lane streaming copy), read + write
    bytes per second, best of 5: the practical HBM ceiling beside the 8 TB/s
    spec."""
    import torch
    from paper_2005_04091_amd import spconv
    n = 512 * 1024 * 1024 // 4
    src = torch.ones((1, 1, 8192, n // 8192), dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    stream = torch.cuda.current_stream(dev)
    best = None
    for _ in range(6):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        spconv.spconv_pad_input(src, 0, out=dst, stream=stream)
        e1.record(stream)
        torch.cuda.synchronize()
        t = e0.elapsed_time(e1)
        best = t if best is None else min(best, t)
    del src, dst
    return 2.0 * n * 4 / (best * 1e-3) / 1e9


def roof(flops, nbytes, ms, peak_tflops):
    """Roofline figures of one launch: fraction of the HBM peak and of the
    arithmetic peak achieved; the most HBM fraction the layer can show at all
    (its bytes over the time of the binding roof: below 1 when the arithmetic
    peak binds first); and the fraction of that binding roof achieved."""
    t = ms * 1e-3
    t_hbm = nbytes / (HBM_PEAK_GBS * 1e9)
    t_alu = flops / (peak_tflops * 1e12)
    t_min = max(t_hbm, t_alu)
    return {
        "hbm_frac": round(nbytes / t / 1e9 / HBM_PEAK_GBS, 4),
        "compute_frac": round(flops / t / 1e12 / peak_tflops, 4),
        "compute_peak_tflops": peak_tflops,
        "max_hbm_frac_at_compute_peak": round(t_hbm / t_min, 4),
        "binding_roof": "hbm" if t_hbm >= t_alu else "compute",
        "binding_roof_frac": round(t_min / t, 4),
    }


def cpu_baseline(layer, budget_s: float, nthreads: int = 0):
    """Time the CPU oracle (as it stands) on a bounded sample of the same layer.

    If the whole layer takes less than the budget, whole-layer passes are
    repeated until the budget is spent and the median pass is reported;
    otherwise a random subset of output planes (n, k) sized to the budget runs
    once. Threads: `nthreads`, or the OpenMP default of this process (0)."""
    import numpy as np
    import oracle

    N, C, H, W, K, R, S = layer.shape
    orc = oracle.get()
    threads = nthreads if nthreads > 0 else orc.max_threads()
    total = N * K
    Hp, Wp = H + 2 * layer.pad, W + 2 * layer.pad
    Ho = (Hp - R) // layer.stride + 1
    Wo = (Wp - S) // layer.stride + 1
    row_nnz = (layer.mask.reshape(K, -1) != 0).sum(1)

    def run(pairs):
        t0 = time.perf_counter()
        orc.conv(layer.x, layer.w, layer.mask, layer.bias, layer.stride, layer.pad, layer.relu, layer.pool,
                 pairs=pairs, nthreads=nthreads)
        return time.perf_counter() - t0

    rng = np.random.default_rng(0)
    order = rng.permutation(total)
    probe = max(threads, 8)
    per_plane = run([(int(p // K), int(p % K)) for p in order[:probe]]) / probe
    if per_plane * total <= budget_s:
        times = []
        spent = 0.0
        while spent < budget_s or not times:
            t = run(None)
            times.append(t)
            spent += t
        dt = statistics.median(times)
        flops = 2.0 * float(row_nnz.sum()) * N * Ho * Wo
        sample = f"the whole layer ({total} output planes), {len(times)} passes, median pass {dt:.2f} s"
    else:
        count = int(min(total, max(probe, budget_s / max(per_plane, 1e-9))))
        pairs = [(int(p // K), int(p % K)) for p in order[:count]]
        dt = run(pairs)
        flops = sum(2.0 * row_nnz[k] * Ho * Wo for _, k in pairs)
        sample = f"{count} of {total} output planes (n, k) of the same layer, chosen at random; {dt:.1f} s"
    return {"value": flops / dt / 1e9, "unit": "GFLOP/s", "cores": threads, "kind": "oracle", "sample": sample}


BLOCK_ROUNDS = 5


def bench_block(args, dev):
    """A chained block per step, with inputs resident in HBM: layer 1 forms its
    input's zero border in the kernel when its rows are wide enough (else one
    pad pass comes first) and writes layer 2's padded input directly (zero
    border); the ResNet shortcut is the unpadded block input. Timed right
    after, on the same buffers: the same chain after a pad pass, both layers
    padding in the kernel (two launches), and the unfused block (a pad pass
    before each layer)."""
    import torch

    from paper_2005_04091_amd import spconv, synth

    if args.workload == "resize_block":
        return bench_resize_block(args, dev)
    x, l1, l2 = synth.make_vgg_block() if args.workload == "vgg_block" else synth.make_resnet_block()
    resnet = args.workload == "resnet_block"
    N, C, H, W, K, R, S = l1.shape
    L1 = spconv.SparseConvLayer(l1.w, l1.mask, l1.bias, H, W, 1, 1, True, False, device=dev)
    L2 = spconv.SparseConvLayer(l2.w, l2.mask, l2.bias, H, W, 1, 1, True, l2.pool, device=dev)
    xd = torch.from_numpy(x).to(dev)
    xp = torch.empty((N, C, H + 2, W + 2), dtype=torch.float32, device=dev)
    y1 = torch.empty((N, K, H, W), dtype=torch.float32, device=dev)
    y1p = torch.empty((N, K, H + 2, W + 2), dtype=torch.float32, device=dev)
    y2 = torch.empty((N, K, L2.Ho, L2.Wo), dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream(dev)
    res = dict(residual=xp, residual_pad=1) if resnet else {}

    def chained_out_pad():
        L1.pad_input(xd, out=xp, stream=stream)
        L1.forward_padded(xp, out=y1p, stream=stream, out_pad=1)
        L2.forward_padded(y1p, out=y2, stream=stream, **res)

    res_unpadded = dict(residual=xd, residual_pad=0) if resnet else {}
    l1_in_kernel = L1.pads_in_kernel(N)

    def fused():
        # Layer 1 pads its input in the kernel when its rows are wide enough,
        # else after one pad pass; it writes layer 2's zero-bordered input.
        if l1_in_kernel:
            L1.forward(xd, out=y1p, stream=stream, out_pad=1)
            L2.forward_padded(y1p, out=y2, stream=stream, **res_unpadded)
        else:
            chained_out_pad()

    def all_in_kernel():
        L1.forward(xd, out=y1, stream=stream, pad_in_kernel=True)
        L2.forward(y1, out=y2, stream=stream, pad_in_kernel=True, **res_unpadded)

    def unfused():
        L1.pad_input(xd, out=xp, stream=stream)
        L1.forward_padded(xp, out=y1, stream=stream)
        L2.pad_input(y1, out=y1p, stream=stream)
        L2.forward_padded(y1p, out=y2, stream=stream, **res)

    def timed(step):
        for _ in range(args.warmup):
            step()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(args.steps):
            step()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / args.steps

    # The variants are timed in rounds, in rotating order, and each reports
    # its median round: whichever runs first after the others would otherwise
    # carry the clock and cache state they leave behind.
    variants = [fused, chained_out_pad, all_in_kernel, unfused]
    times = [[] for _ in variants]
    for r in range(BLOCK_ROUNDS):
        for i in range(len(variants)):
            j = (i + r) % len(variants)
            times[j].append(timed(variants[j]))
    ms, ms_chained, ms_in_kernel, ms_unfused = (statistics.median(t) for t in times)
    nnz1, nnz2 = L1.host_csr.nnz, L2.host_csr.nnz
    flops = 2.0 * (nnz1 + nnz2) * N * H * W
    rec = {
        "metric": "ms/layer + nonzero GFLOP/s + % HBM roofline, fused sparse conv, 1 MI355X",
        "value": round(flops / (ms * 1e-3) / 1e9, 2),
        "unit": "GFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic (seeded Bernoulli-masked weights U[-1,1), input U[0,1), bias U[-0.1,0.1))",
        "config": {"workload": BLOCKS[args.workload], "N": N, "C": C, "K": K, "H": H, "W": W,
                   "nnz": [nnz1, nnz2], "pool": bool(l2.pool), "residual": resnet},
        "ms_per_step_unfused": round(ms_unfused, 5),
        "ms_per_step_chained_out_pad": round(ms_chained, 5),
        "ms_per_step_both_pad_in_kernel": round(ms_in_kernel, 5),
        "layer1_pads_in_kernel": l1_in_kernel,
        "fusion_saving_frac": round(1.0 - ms / ms_unfused, 4),
        "timing": f"median of {BLOCK_ROUNDS} rounds of {args.steps} steps per variant, variants in rotating order",
    }
    print(json.dumps(rec), flush=True)


def _timed(args, stream, step):
    import torch
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(args.steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / args.steps


def bench_resize_block(args, dev):
    """Resize-Conv-ReLU-Maxpool per step, source resident in HBM: the resize
    writes the conv's padded input directly (one pass), then the fused conv +
    bias + ReLU + max-pool. `unfused` resizes into a plain tensor and pads it
    in a second pass before the same conv. The resize kernel is also timed on
    its own, against its algorithmic bytes (source taps read once, padded
    output written once)."""
    import torch

    from paper_2005_04091_amd import spconv, synth

    src, layer = synth.make_resize_block()
    N, C, H, W, K, R, S = layer.shape
    Hin, Win = int(src.shape[2]), int(src.shape[3])
    L = spconv.SparseConvLayer(layer.w, layer.mask, layer.bias, H, W, 1, 1, True, True, device=dev)
    sd = torch.from_numpy(src).to(dev)
    xr = torch.empty((N, C, H, W), dtype=torch.float32, device=dev)
    xp = torch.empty((N, C, H + 2, W + 2), dtype=torch.float32, device=dev)
    y = torch.empty((N, K, L.Ho, L.Wo), dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream(dev)

    def fused():
        L.resize_pad_input(sd, out=xp, stream=stream)
        L.forward_padded(xp, out=y, stream=stream)

    def unfused():
        spconv.spconv_resize_pad_input(sd, H, W, 0, out=xr, stream=stream)
        L.pad_input(xr, out=xp, stream=stream)
        L.forward_padded(xp, out=y, stream=stream)

    def resize_only():
        L.resize_pad_input(sd, out=xp, stream=stream)

    variants = [fused, unfused, resize_only]
    times = [[] for _ in variants]
    for r in range(BLOCK_ROUNDS):
        for i in range(len(variants)):
            j = (i + r) % len(variants)
            times[j].append(_timed(args, stream, variants[j]))
    ms, ms_unfused, ms_resize = (statistics.median(t) for t in times)
    nnz = L.host_csr.nnz
    flops = 2.0 * nnz * N * H * W
    rbytes = resize_source_bytes(N * C, Hin, Win, H, W) + 4.0 * N * C * (H + 2) * (W + 2)
    rec = {
        "metric": "ms/layer + nonzero GFLOP/s + % HBM roofline, fused sparse conv, 1 MI355X",
        "value": round(flops / (ms * 1e-3) / 1e9, 2),
        "unit": "GFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic (seeded Bernoulli-masked weights U[-1,1), source U[0,1), bias U[-0.1,0.1))",
        "config": {"workload": BLOCKS[args.workload], "N": N, "C": C, "K": K, "Hin": Hin, "Win": Win, "H": H,
                   "W": W, "nnz": nnz, "pool": True},
        "ms_per_step_unfused": round(ms_unfused, 5),
        "fusion_saving_frac": round(1.0 - ms / ms_unfused, 4),
        "timing": f"median of {BLOCK_ROUNDS} rounds of {args.steps} steps per variant, variants in rotating order",
        "resize_kernel": {"ms": round(ms_resize, 5), "algorithmic_bytes": rbytes,
                          "GB/s": round(rbytes / (ms_resize * 1e-3) / 1e9, 1),
                          "hbm_frac": round(rbytes / (ms_resize * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)},
    }
    if args.copy_calibration:
        copy_calibration(args.copy_calibration, dev)
    print(json.dumps(rec), flush=True)


METRIC = "ms/layer + nonzero GFLOP/s + % HBM roofline, fused sparse conv, 1 MI355X"
DATA = "synthetic (seeded Bernoulli-masked weights U[-1,1), input U[0,1), bias U[-0.1,0.1))"
COLD_REPS = 30  # the paper reports the median of 30 runs (--cold-reps changes it for profiling runs)


def layer_launch(L, x, out, stream, xp=None):
    """The forward of one layer on a resident batch, as the step runs it: one
    launch on the unpadded input when the kernel forms the zero border while
    staging (wide rows), else the forward on an already padded copy `xp`."""
    N = int(x.shape[0])
    if L.pads_in_kernel(N):
        return lambda: L.forward(x, out=out, stream=stream)
    return lambda: L.forward_padded(xp, out=out, stream=stream)


def per_config_record(name, args, dev, stream):
    """One of the other layer configurations, measured like the block's layers:
    back-to-back launches (warm), the cold median of 30 of the forward alone and
    of pad + forward, nonzero GFLOP/s, and the roofline figures against HBM and
    the arithmetic peak of the path that runs (v_fma_f32 for the sparse kernels,
    the fp32 matrix cores for the dense one)."""
    import torch
    from paper_2005_04091_amd import spconv, synth
    layer = synth.make_layer(name)
    N, C, H, W, K, R, S = layer.shape
    L = spconv.SparseConvLayer(layer.w, layer.mask, layer.bias, H, W, layer.stride, layer.pad, layer.relu,
                               layer.pool, device=dev, path="auto", N=N)
    x = torch.from_numpy(layer.x).to(dev)
    xp = torch.empty((N, C, H + 2 * layer.pad, W + 2 * layer.pad), dtype=torch.float32, device=dev)
    out = torch.empty((N, K, L.Ho, L.Wo), dtype=torch.float32, device=dev)
    fused_pad = L.pads_in_kernel(N)
    if not fused_pad:
        L.pad_input(x, out=xp, stream=stream)
    fwd = layer_launch(L, x, out, stream, xp)

    def step():
        if not fused_pad:
            L.pad_input(x, out=xp, stream=stream)
        fwd()

    ms_warm = _timed(args, stream, fwd)
    ms_cold = cold_median_ms(fwd, stream, args.cold_reps, dev)
    ms_step_cold = cold_median_ms(step, stream, args.cold_reps, dev)
    nnz = L.host_csr.nnz
    flops, nbytes, _ = algorithmic(layer, nnz)
    if fused_pad:
        nbytes -= 4.0 * N * C * ((H + 2 * layer.pad) * (W + 2 * layer.pad) - H * W)
    rec = {"workload": name, "description": WORKLOADS[name], "path": L.path, "nnz": nnz,
           "density": round(nnz / (K * C * R * S), 5), "pad": "in the kernel" if fused_pad else "separate pass",
           "plan": L.plan(N, unpadded=fused_pad),
           "ms_per_layer": round(ms_cold, 5), "ms_per_layer_warm": round(ms_warm, 5),
           "ms_per_layer_with_pad": round(ms_step_cold, 5),
           "nonzero_gflops": round(flops / (ms_cold * 1e-3) / 1e9, 1),
           "nonzero_gflops_warm": round(flops / (ms_warm * 1e-3) / 1e9, 1),
           "algorithmic_bytes": int(nbytes), "nonzero_flops": flops}
    if L.path == "dense":
        dflops = 2.0 * K * C * R * S * N * L.Ho * L.Wo
        nbytes_d = nbytes + 4.0 * L.dense.numel() - 8.0 * nnz
        rec["roof"] = roof(dflops, nbytes_d, ms_cold, MFMA_FP32_TFLOPS)
        rec["roof"]["flops_counted"] = "dense filter work on the fp32 matrix cores"
        rec["nonzero_flops_roof"] = roof(flops, nbytes, ms_cold, VALU_FP32_FMA_TFLOPS)
    else:
        rec["roof"] = roof(flops, nbytes, ms_cold, VALU_FP32_FMA_TFLOPS)
        rec["roof"]["flops_counted"] = "nonzero multiply-adds on v_fma_f32"
    return rec


def cpu_baseline_block(layers, budget_s: float):
    """The CPU oracle (as it stands) on the block's two layers: whole-block
    passes repeated while they fit the budget (median pass), else the same
    random share of output planes of each layer. Layer 2 runs on its own
    seeded input of the block's shape (the oracle's cost does not depend on
    the values)."""
    import numpy as np
    import oracle
    orc = oracle.get()
    threads = orc.max_threads()
    rng = np.random.default_rng(0)
    per = []
    for layer in layers:
        N, C, H, W, K, R, S = layer.shape
        probe = max(threads, 8)
        pairs = [(int(p // K), int(p % K)) for p in rng.permutation(N * K)[:probe]]
        t0 = time.perf_counter()
        orc.conv(layer.x, layer.w, layer.mask, layer.bias, layer.stride, layer.pad, layer.relu, layer.pool, pairs=pairs)
        per.append((time.perf_counter() - t0) / probe)
    whole = sum(pp * l.shape[0] * l.shape[4] for pp, l in zip(per, layers))
    row_nnz = [(l.mask.reshape(l.shape[4], -1) != 0).sum(1) for l in layers]

    def flops_of(layer, rn, pairs):
        N, C, H, W, K, R, S = layer.shape
        if pairs is None:
            return 2.0 * float(rn.sum()) * N * H * W
        return sum(2.0 * rn[k] * H * W for _, k in pairs)

    if whole <= budget_s / 2:
        times = []
        while sum(times) < budget_s or not times:
            t0 = time.perf_counter()
            for layer in layers:
                orc.conv(layer.x, layer.w, layer.mask, layer.bias, layer.stride, layer.pad, layer.relu, layer.pool)
            times.append(time.perf_counter() - t0)
        dt = statistics.median(times)
        flops = sum(flops_of(l, rn, None) for l, rn in zip(layers, row_nnz))
        sample = f"the whole block (both layers), {len(times)} passes, median pass {dt:.2f} s"
    else:
        share = budget_s / whole
        dt = 0.0
        flops = 0.0
        planes = 0
        for layer, rn in zip(layers, row_nnz):
            N, K = layer.shape[0], layer.shape[4]
            count = max(threads, int(share * N * K))
            pairs = [(int(p // K), int(p % K)) for p in rng.permutation(N * K)[:count]]
            t0 = time.perf_counter()
            orc.conv(layer.x, layer.w, layer.mask, layer.bias, layer.stride, layer.pad, layer.relu, layer.pool,
                     pairs=pairs)
            dt += time.perf_counter() - t0
            flops += flops_of(layer, rn, pairs)
            planes += count
        sample = (f"{planes} random output planes (n, k) of the block's two layers "
                  f"({100 * share:.0f}% of each), {dt:.1f} s")
    return {"value": round(flops / dt / 1e9, 3), "unit": "GFLOP/s", "cores": threads, "kind": "oracle",
            "sample": sample}


def bench_vgg(args, dev):
    """The VGG-style block, the default workload (see the module docstring)."""
    import torch
    from paper_2005_04091_amd import spconv, synth

    x, l1, l2 = synth.make_vgg_block()
    N, C, H, W, K, R, S = l1.shape
    print(f"[bench] VGG block N={N} C={C} K={K} {H}x{W}", file=sys.stderr, flush=True)
    L1 = spconv.SparseConvLayer(l1.w, l1.mask, l1.bias, H, W, 1, 1, True, False, device=dev)
    L2 = spconv.SparseConvLayer(l2.w, l2.mask, l2.bias, H, W, 1, 1, True, True, device=dev)
    assert L1.path == L2.path == "sparse"
    xd = torch.from_numpy(x).to(dev)
    xp = torch.empty((N, C, H + 2, W + 2), dtype=torch.float32, device=dev)
    y1p = torch.empty((N, K, H + 2, W + 2), dtype=torch.float32, device=dev)
    y2 = torch.empty((N, K, L2.Ho, L2.Wo), dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream(dev)
    in_kernel = L1.pads_in_kernel(N)
    if not in_kernel:
        L1.pad_input(xd, out=xp, stream=stream)
    plans = [L1.plan(N, unpadded=in_kernel), L2.plan(N)]
    print(f"[bench] plans {plans}, layer 1 pads in the kernel: {in_kernel}", file=sys.stderr, flush=True)

    def conv1():
        if in_kernel:
            L1.forward(xd, out=y1p, stream=stream, out_pad=1)
        else:
            L1.forward_padded(xp, out=y1p, stream=stream, out_pad=1)

    def conv2():
        L2.forward_padded(y1p, out=y2, stream=stream)

    def step():
        if not in_kernel:
            L1.pad_input(xd, out=xp, stream=stream)
        conv1()
        conv2()

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    # Timed steps: one event pair around the K steps. An event recorded
    # between two kernels holds the second back until the first has drained
    # and signalled, so the per-kernel durations the roofline uses come from
    # a second pass of K steps with events around each kernel.
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0.record(stream)
    for _ in range(args.steps):
        step()
    t1.record(stream)
    torch.cuda.synchronize()
    ms_per_step = t0.elapsed_time(t1) / args.steps
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    for i in range(args.steps):
        if not in_kernel:
            L1.pad_input(xd, out=xp, stream=stream)
        ev[i][0].record(stream)
        conv1()
        ev[i][1].record(stream)
        conv2()
        ev[i][2].record(stream)
    torch.cuda.synchronize()
    ms1 = statistics.mean(e[0].elapsed_time(e[1]) for e in ev)
    ms2 = statistics.mean(e[1].elapsed_time(e[2]) for e in ev)
    print(f"[bench] step {ms_per_step:.4f} ms, conv1 {ms1:.4f} ms, conv2+pool {ms2:.4f} ms", file=sys.stderr,
          flush=True)
    cold1 = cold_median_ms(conv1, stream, args.cold_reps, dev)
    cold2 = cold_median_ms(conv2, stream, args.cold_reps, dev)
    copy_gbs = measured_copy_gbs(dev)

    nnz1, nnz2 = L1.host_csr.nnz, L2.host_csr.nnz
    f1, b1, _ = algorithmic(l1, nnz1)
    f2, b2, _ = algorithmic(l2, nnz2)
    if in_kernel:  # layer 1 reads the unpadded input
        b1 -= 4.0 * N * C * ((H + 2) * (W + 2) - H * W)
    b1 += 4.0 * N * K * ((H + 2) * (W + 2) - H * W)  # it also writes layer 2's zero border
    flops = f1 + f2
    layers = {
        "conv1": {"ms_per_layer": round(cold1, 5), "ms_in_step": round(ms1, 5), "nnz": nnz1, "plan": plans[0],
                  "nonzero_gflops": round(f1 / (cold1 * 1e-3) / 1e9, 1), "algorithmic_bytes": int(b1),
                  "nonzero_flops": f1, "roof": roof(f1, b1, cold1, VALU_FP32_FMA_TFLOPS),
                  "pad": "formed in the kernel while staging" if in_kernel else "separate pass"},
        "conv2_pool": {"ms_per_layer": round(cold2, 5), "ms_in_step": round(ms2, 5), "nnz": nnz2, "plan": plans[1],
                       "nonzero_gflops": round(f2 / (cold2 * 1e-3) / 1e9, 1), "algorithmic_bytes": int(b2),
                       "nonzero_flops": f2, "roof": roof(f2, b2, cold2, VALU_FP32_FMA_TFLOPS),
                       "pad": "its input is layer 1's zero-bordered output"},
    }
    dom, fd, bd, msd = ("conv1", f1, b1, ms1) if ms1 >= ms2 else ("conv2_pool", f2, b2, ms2)
    achieved = fd / (msd * 1e-3) / 1e12
    inst = layers[dom]["plan"]
    kname = (f"spconv_s1_kernel<{inst['pixels_per_lane']}, {inst['images_per_group']}, "
             f"{inst['channels_per_wave']}, {'true' if dom == 'conv2_pool' else 'false'}>")
    traffic = measured_traffic(f"vgg_{dom}", "fwd")
    rec = {
        "metric": METRIC,
        "value": round(flops / (ms_per_step * 1e-3) / 1e9, 2),
        "unit": "GFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": DATA + "; channels 3..63 of the block input are zero",
        "config": {"workload": BLOCKS["vgg_block"], "N": N, "C": C, "K": K, "H": H, "W": W, "R": R, "S": S,
                   "nnz": [nnz1, nnz2], "density": 0.2, "pool": "layer 2", "path": "sparse"},
        "ms_per_layer": {k: v["ms_per_layer"] for k, v in layers.items()},
        "ms_per_layer_protocol": f"median of {args.cold_reps} runs, each after a 512 MiB write that flushes the "
                                 "last-level cache; HIP events around the forward alone",
        "layers": layers,
        "hbm_copy_measured_GBs": round(copy_gbs, 1),
        "roofline": {
            "kernel": kname,
            "layer": dom,
            "bound": "alu",
            "achieved": round(achieved, 3),
            "peak": VALU_FP32_FMA_TFLOPS,
            "unit": "TFLOP/s",
            "frac": round(achieved / VALU_FP32_FMA_TFLOPS, 4),
            "traffic": traffic,
            "traffic_source": f"profiles/spconv_fwd_vgg_{dom}_traffic.json (counter runs, source hash checked)"
                              if traffic is not None else None,
            "algorithmic_bytes": int(bd),
            "flops": fd,
            "ms_per_launch": round(msd, 5),
            "timing": "HIP events on the launch stream around this kernel in each of K steps run after the timed ones, mean",
        },
        "hbm_bar": {
            "target_frac": 0.5,
            "note": "at 78.6 TFLOP/s (v_fma_f32, packed FP32 disabled) a layer of F nonzero FLOPs and B bytes "
                    "cannot take less than F/78.6 TF, so its HBM fraction is at most (B/8 TB/s)/(F/78.6 TF)",
            "max_hbm_frac_at_fma_peak": {k: v["roof"]["max_hbm_frac_at_compute_peak"] for k, v in layers.items()},
        },
    }
    if not args.no_per_config:
        pc = []
        for name in ("tiny", "resnet", "conv_pool", "narrow_d0.05", "narrow_d0.2", "narrow_d0.5"):
            print(f"[bench] per-config {name}", file=sys.stderr, flush=True)
            pc.append(per_config_record(name, args, dev, stream))
        rec["per_config"] = pc
        rec["hbm_bar"]["max_hbm_frac_at_fma_peak"].update(
            {r["workload"]: r["roof"]["max_hbm_frac_at_compute_peak"] for r in pc})
    if args.copy_calibration:
        copy_calibration(args.copy_calibration, dev)
    if not args.no_cpu_baseline:
        print("[bench] timing the CPU oracle on the block", file=sys.stderr, flush=True)
        rec["cpu_baseline"] = cpu_baseline_block([l1, l2], args.cpu_budget)
    print(json.dumps(rec), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="vgg_block", choices=sorted(WORKLOADS) + sorted(BLOCKS),
                    help="vgg_block (default): the chained VGG block with per-config records; with --compare, "
                         "its fused and unfused variants instead; other names: one layer or block")
    ap.add_argument("--cpu-budget", type=float, default=15.0, help="seconds of oracle work for cpu_baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cold-reps", type=int, default=COLD_REPS,
                    help="runs per cache-flushed median (30, as the paper's medians; fewer for counter runs)")
    ap.add_argument("--no-per-config", action="store_true",
                    help="default workload only: leave out the per-config records of the other layers")
    ap.add_argument("--cold", action="store_true",
                    help="also report the forward's median over 30 runs with the last-level cache flushed before each")
    ap.add_argument("--compare", action="store_true",
                    help="also time the step with a separate pad pass and with the pad formed in the kernel")
    ap.add_argument("--path", default="auto", choices=["auto", "sparse", "dense"],
                    help="kernel family; auto = the library's break-even-density dispatcher")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="after timing, copy MIB MiB device-to-device three times (counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU: this build runs on a single MI355X and has no multi-GPU path "
              f"(asked for --gpus {args.gpus}).", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2005_04091_amd import spconv, synth

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    # No cyclic garbage collection while launches are timed: a full pass over
    # the interpreter's objects (tens of ms with torch loaded) stalls the host
    # between two launches and lands inside the events' window (a 47 ms gap
    # between two back-to-back launches was seen in a kernel trace).
    gc.collect()
    gc.disable()
    dev = torch.device("cuda:0")
    if args.workload == "vgg_block" and not args.compare:
        bench_vgg(args, dev)
        return
    if args.workload in BLOCKS:
        bench_block(args, dev)
        return
    layer = synth.make_layer(args.workload)
    N, C, H, W, K, R, S = layer.shape
    print(f"[bench] workload {args.workload}: {WORKLOADS[args.workload]}", file=sys.stderr, flush=True)
    L = spconv.SparseConvLayer(layer.w, layer.mask, layer.bias, H, W, layer.stride, layer.pad, layer.relu,
                               layer.pool, device=dev, path=args.path, N=N)
    nnz = L.host_csr.nnz
    dense = L.path == "dense"
    print(f"[bench] path {L.path}: {L.plan(N, unpadded=L.pads_in_kernel(N))}", file=sys.stderr, flush=True)
    x = torch.from_numpy(layer.x).to(dev)
    xp = torch.empty((N, C, H + 2 * layer.pad, W + 2 * layer.pad), dtype=torch.float32, device=dev)
    out = torch.empty((N, K, L.Ho, L.Wo), dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream(dev)

    # A step is the whole path on one batch. When the layer's kernel forms the
    # zero border while staging its input (stride-1 and dense kernels), that is
    # one launch on the unpadded input; otherwise the pad pass, then the
    # forward on the padded copy.
    fused_pad = L.pads_in_kernel(N)

    def step():
        if fused_pad:
            L.forward(x, out=out, stream=stream)
        else:
            L.pad_input(x, out=xp, stream=stream)
            L.forward_padded(xp, out=out, stream=stream)

    def separate_pad_step():
        L.pad_input(x, out=xp, stream=stream)
        L.forward_padded(xp, out=out, stream=stream)

    def timed(fn):
        for _ in range(args.warmup):
            fn()
        torch.cuda.synchronize()
        t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t0.record(stream)
        for _ in range(args.steps):
            fn()
        t1.record(stream)
        torch.cuda.synchronize()
        return t0.elapsed_time(t1) / args.steps

    ms_per_step = timed(step)
    ms_separate = ms_in_kernel = None
    if args.compare:  # other launch configurations of the same kernels (kept out of default runs and profiles)
        ms_separate = timed(separate_pad_step)
        if L.can_pad_in_kernel(N):
            ms_in_kernel = timed(lambda: L.forward(x, out=out, stream=stream, pad_in_kernel=True))
    pad_only = timed(lambda: L.pad_input(x, out=xp, stream=stream))
    # Average duration of one forward launch for the roofline: the kernel the
    # step runs, launched back to back on the same stream, one event pair
    # around all launches, so that per-launch event and dispatch gaps do not
    # count (with a separate pad pass: the forward on the padded input).
    fwd_avg = timed((lambda: L.forward(x, out=out, stream=stream)) if fused_pad
                    else (lambda: L.forward_padded(xp, out=out, stream=stream)))

    # The same forward with a cold last-level cache (median of 30, as the paper
    # reports medians), and the measured copy ceiling.
    fwd_fn = (lambda: L.forward(x, out=out, stream=stream)) if fused_pad \
        else (lambda: L.forward_padded(xp, out=out, stream=stream))
    fwd_cold = cold_median_ms(fwd_fn, stream, 30, dev) if args.cold else None
    copy_gbs = measured_copy_gbs(dev)

    flops, fwd_bytes, pad_bytes = algorithmic(layer, nnz)
    if fused_pad:  # the kernel reads the unpadded input
        fwd_bytes -= 4.0 * N * C * ((H + 2 * layer.pad) * (W + 2 * layer.pad) - H * W)
    value = flops / (ms_per_step * 1e-3) / 1e9
    if dense:
        # The dense kernel's algorithmic work is every filter tap (its FLOPs on
        # the stored pixels), on the fp32 matrix cores; its filter read is the
        # packed dense array instead of the CSR.
        kern_flops = 2.0 * K * C * R * S * N * (H + 2 * layer.pad - R + 1) * (W + 2 * layer.pad - S + 1)
        fwd_bytes += 4.0 * L.dense.numel() - (8.0 * nnz)
        bound, peak, kname = "mfma", MFMA_FP32_TFLOPS, "spconv_dense_kernel"
    else:
        kern_flops = flops
        bound, peak, kname = "alu", VALU_FP32_FMA_TFLOPS, "spconv_fwd_kernel"
    achieved_tflops = kern_flops / (fwd_avg * 1e-3) / 1e12
    rec = {
        "metric": "ms/layer + nonzero GFLOP/s + % HBM roofline, fused sparse conv, 1 MI355X",
        "value": round(value, 2),
        "unit": "GFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic (seeded Bernoulli-masked weights U[-1,1), input U[0,1), bias U[-0.1,0.1))",
        "config": {"workload": WORKLOADS[args.workload], "N": N, "C": C, "K": K, "H": H, "W": W, "R": R, "S": S,
                   "stride": layer.stride, "pad": layer.pad, "pool": layer.pool, "nnz": nnz,
                   "density": round(nnz / (K * C * R * S), 5), "path": L.path, "pad": "fused" if fused_pad else "separate"},
        "ms_per_layer": round(fwd_avg, 5),
        "pad": "in the kernel's LDS staging" if fused_pad else "separate pass",
        "ms_per_step_separate_pad": None if ms_separate is None else round(ms_separate, 5),
        "ms_per_step_pad_in_kernel": None if ms_in_kernel is None else round(ms_in_kernel, 5),
        "ms_pad_pass": round(pad_only, 5),
        "nonzero_gflops_layer": round(flops / (fwd_avg * 1e-3) / 1e9, 2),
        "hbm_roofline_frac": round(fwd_bytes / (fwd_avg * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
        "ms_per_layer_cold_median": None if fwd_cold is None else round(fwd_cold, 5),
        "hbm_copy_measured_GBs": round(copy_gbs, 1),
        "hbm_frac_of_measured_copy": round(fwd_bytes / (fwd_avg * 1e-3) / 1e9 / copy_gbs, 4),
        "roofline": {
            "kernel": kname,
            "bound": bound,
            "achieved": round(achieved_tflops, 3),
            "peak": peak,
            "unit": "TFLOP/s",
            "frac": round(achieved_tflops / peak, 4),
            "traffic": measured_traffic(args.workload, "dense" if dense else "fwd"),
            "algorithmic_bytes": int(fwd_bytes),
            "flops": kern_flops,
        },
    }
    if args.copy_calibration:
        copy_calibration(args.copy_calibration, dev)
    if not args.no_cpu_baseline:
        print("[bench] timing the CPU oracle", file=sys.stderr, flush=True)
        cb = cpu_baseline(layer, args.cpu_budget)
        cb["value"] = round(cb["value"], 3)
        rec["cpu_baseline"] = cb
        cb1 = cpu_baseline(layer, args.cpu_budget / 2, nthreads=1)
        cb1["value"] = round(cb1["value"], 3)
        rec["cpu_baseline_1thread"] = cb1
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
