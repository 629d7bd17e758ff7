"""Benchmark of the 1-bit FQT layer backward on one MI355X.

Workload: VGG-16 CIFAR-shaped 3x3 convolution 256 -> 256 on 8x8 maps, batch 128,
fp32 X / W / dY (dY per-sample lognormal(0, 2) scale with 13 of 128 samples x100),
AGP Bernoulli keeping 1/4 of the groups (b = 4), Philox seed 0.  A step is one
fqt_layer_backward: group statistics, AGP selection, SR + bit-plane packing,
sign packing of X (bit-im2col) and W, and both binary products with rescale.

Prints one JSON line: throughput in binary TOPS (2 x D*C*k*k*N*Ho*Wo binary
multiply-accumulates per product, both products, per step time), the roofline
of the dominant kernel timed with HIP events on its own stream, and the CPU
oracle timed on a bounded sample on the host.
"""
import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

WORKLOAD = "vgg_cifar_conv3x3_256"
HBM_PEAK_GBS = 8000.0
# Integer VALU issue rate: 256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz lane-instructions/s.
VALU_LANE_OPS = 256 * 4 * 16 * 2.4e9
# Popcount engine: one 64-bit AND + popcount-accumulate is 4 lane-instructions
# (2 v_and_b32, 2 v_bcnt_u32_b32) for 64 binary MACs = 128 binary ops.
POPC_PEAK_TOPS = VALU_LANE_OPS * 128 / 4 / 1e12


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=200)
    p.add_argument("--warmup", type=int, default=20)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-seconds", type=float, default=12.0,
                   help="bound on the CPU oracle sample (seconds of work)")
    p.add_argument("--no-graph", action="store_true", help="time eager launches only")
    return p.parse_args()


def cpu_baseline(x, w, dy, layer, wl, ops_per_step, budget_s):
    """The oracle, as it stands, on the host cores: full layer backward repeated until
    about `budget_s` seconds of work have been done (at least once)."""
    from threadpoolctl import threadpool_info

    from oracle import fqt as ofqt
    reps, t0 = 0, time.perf_counter()
    while True:
        ofqt.layer_backward(x, w, dy, wl.bits, wl.agp_mode, seed=wl.philox_seed,
                            stride=layer.stride, pad=layer.pad)
        reps += 1
        el = time.perf_counter() - t0
        if el >= budget_s:
            break
    threads = max([1] + [int(i.get("num_threads", 1)) for i in threadpool_info()])
    return {"value": ops_per_step * reps / el / 1e12, "unit": "TOPS", "cores": threads,
            "kind": "oracle",
            "sample": f"{reps} full layer backward(s) of {WORKLOAD} in {el:.1f} s "
                      f"({el / reps * 1e3:.0f} ms each; numpy, BLAS threads={threads})"}


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this benchmark runs on one GPU only; the layer backward "
                                   "shards by data parallelism with one dW all-reduce, which "
                                   "is not part of this build", "n_gpus": args.gpus}))
        sys.exit(2)

    import torch

    from paper_2408_14267_amd import fqt
    from paper_2408_14267_amd.workloads import WORKLOADS, draw_layer

    wl = WORKLOADS[WORKLOAD]
    layer = wl.layers[0]
    dev = torch.device("cuda:0")
    x, w, dy = draw_layer(layer, wl.recipe, wl.seed, wl.dtype)
    X, W, dY = (torch.from_numpy(a).to(dev) for a in (x, w, dy))
    dX, dW = torch.empty_like(X), torch.empty_like(W)
    desc = fqt.layer_desc(layer)
    cfg = fqt.quant_cfg(wl.bits, wl.agp_mode, wl.philox_seed, 0, 0)
    ws = fqt.workspace(desc, cfg, device=dev)
    stream = torch.cuda.current_stream()
    macs = layer.binary_macs()
    ops_per_step = 2 * 2 * macs            # two products, 2 ops per binary MAC

    def step():
        fqt.fqt_layer_backward(desc, cfg, X, W, dY, dX, dW, ws, stream)

    def timed(fn, k):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(k):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / k

    for _ in range(args.warmup):
        step()
    ms_eager = timed(step, args.steps)

    ms_graph = None
    if not args.no_graph:
        g = torch.cuda.CUDAGraph()
        side = torch.cuda.Stream()
        side.wait_stream(stream)
        with torch.cuda.stream(side):
            step_s = lambda: fqt.fqt_layer_backward(desc, cfg, X, W, dY, dX, dW, ws, side)
            step_s()
            torch.cuda.synchronize()
            with torch.cuda.graph(g, stream=side):
                step_s()
        torch.cuda.synchronize()
        for _ in range(args.warmup):
            g.replay()
        ms_graph = timed(g.replay, args.steps)
    ms = ms_graph if ms_graph is not None else ms_eager

    # Per-product timing of the dominant kernel: the two products are single-kernel
    # entry points; events bracket each launch on the stream it is issued on.
    q = fqt.QGrad(desc, cfg, device=dev)
    qws = fqt.workspace(desc, cfg, fqt.FQT_WS_QUANTIZE, device=dev)
    K = layer.C * layer.kh * layer.kw
    R = layer.N * layer.Ho * layer.Wo
    Wd, Wr = (layer.D + 63) // 64, (R + 63) // 64
    xs = torch.empty(K * Wr, dtype=torch.int64, device=dev)
    xsum = torch.empty(K, dtype=torch.int32, device=dev)
    wsg = torch.empty(K * Wd, dtype=torch.int64, device=dev)
    wsum = torch.empty(K, dtype=torch.int32, device=dev)
    fqt.fqt_agp_scq_quantize(desc, cfg, dY, q, qws, stream)
    fqt.fqt_pack_bits(X, fqt.FQT_F32, 0, 0, 0, fqt.FQT_PACK_IM2COL, desc, xs, xsum, stream)
    fqt.fqt_pack_bits(W, fqt.FQT_F32, layer.D, K, K, fqt.FQT_PACK_ALONG_ROWS, None, wsg, wsum, stream)
    kernels = {
        "gemm_dw": lambda: fqt.fqt_binary_gemm_dw(desc, cfg, q, xs, dW, None, stream),
        "gemm_dx": lambda: fqt.fqt_binary_gemm_dx(desc, cfg, q, wsg, dX, None, stream),
    }
    per = {}
    for name, fn in kernels.items():
        for _ in range(args.warmup):
            fn()
        per[name] = timed(fn, args.steps)
    dom = max(per, key=per.get)
    # Algorithmic binary ops of one product launch (binary-equivalent, as the paper counts).
    achieved = 2 * macs / (per[dom] * 1e-3) / 1e12
    roofline = {"bound": "alu", "achieved": achieved, "peak": POPC_PEAK_TOPS, "unit": "TOPS",
                "frac": achieved / POPC_PEAK_TOPS, "traffic": None, "kernel": dom,
                "kernel_ms": per[dom]}

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(x, w, dy, layer, wl, ops_per_step, args.cpu_seconds)

    out = {
        "metric": "binary backward TOPS + layer-backward ms (VGG16/ResNet18 shapes), % roofline",
        "value": ops_per_step / (ms * 1e-3) / 1e12,
        "unit": "TOPS",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u1",
        "data": "synthetic",
        "config": {"workload": WORKLOAD, "layer": "conv3x3 256->256, 8x8, stride 1, pad 1",
                   "batch": layer.N, "bits": wl.bits, "agp": "bernoulli", "inputs": "f32",
                   "accumulate": "i32", "hip_graph": ms_graph is not None,
                   "ms_per_step_eager": ms_eager, "ms_per_step_graph": ms_graph,
                   "per_kernel_ms": per, "binary_ops_per_step": ops_per_step},
        "roofline": roofline,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out))


if __name__ == "__main__":
    main()
