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
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
MFMA_I8_PEAK_TOPS = 5000.0     # MI355X dense int8 MFMA

# HBM traffic per launch from rocprofv3 counter runs of this benchmark (FETCH_SIZE and
# WRITE_SIZE in KiB per dispatch, one run each), scaled by what the same counters read for
# a 256 MiB device copy in those runs (FETCH_SIZE reads half the copied bytes).  The figures
# are reported only while the kernel sources are byte-identical to the ones they were
# measured on (TRAFFIC_DIGEST: sha256 over the names and contents of every file in csrc/).
FETCH_SCALE = 262144.0 / 131086.7
WRITE_SCALE = 1.0
TRAFFIC_DIGEST = "44a2b213ef2730474d4b393662918398bd0843d8c2cdcf0dcb3d3f939fde34e1"
TRAFFIC = {
    # entry: (FETCH_SIZE KiB, WRITE_SIZE KiB) per launch of its kernels
    "gemm_dx": (2538.0, 8192.0),
    "pack_x": (4143.3, 2304.0),
    "pack_w": (1179.5, 585.0),
}


def sources_digest():
    import hashlib
    d = os.path.join(ROOT, "paper_2408_14267_amd", "csrc")
    h = hashlib.sha256()
    for name in sorted(os.listdir(d)):
        if name.endswith((".hip", ".hpp", ".h", ".cpp")):
            h.update(name.encode())
            with open(os.path.join(d, name), "rb") as f:
                h.update(f.read())
    return h.hexdigest()


def measured_traffic(kernel):
    """HBM bytes per launch of `kernel`, or None when not measured on the current sources."""
    if kernel not in TRAFFIC or sources_digest() != TRAFFIC_DIGEST:
        return None
    fetch_kib, write_kib = TRAFFIC[kernel]
    return (fetch_kib * FETCH_SCALE + write_kib * WRITE_SCALE) * 1024.0


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=200)
    p.add_argument("--warmup", type=int, default=20)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-seconds", type=float, default=12.0,
                   help="bound on the CPU oracle sample (seconds of work)")
    p.add_argument("--no-graph", action="store_true", help="time eager launches only")
    p.add_argument("--suite", choices=("resnet18_32px", "vgg16_224_bf16", "gemm_sweep", "forward",
                                       "table5"),
                   help="instead of the benchmark line: per-layer times of a whole network's "
                        "layer backwards, the dW binary GEMM sweep, the binary forward of "
                        "the VGG CIFAR conv layer and of every ResNet-18 / VGG-16 layer, or "
                        "average-1-bit against 1-bit products at the sizes of the paper's "
                        "Table 5 (one JSON line each)")
    p.add_argument("--calib-copy-mib", type=int, default=0,
                   help="first run a plain device copy of this many MiB (three times), so that "
                        "a counter run can scale FETCH_SIZE / WRITE_SIZE by a known byte count")
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


def _gen(torch, shape, dtype, dev, scale=None):
    x = torch.randn(shape, device=dev, dtype=torch.float32)
    if scale is not None:
        x *= scale
    return x.to(dtype)


def suite(name, reps=10):
    """Per-layer eager times of the layer backward over a whole network (inputs drawn on the
    GPU with the workload's recipe distributions), or the dW binary GEMM sweep."""
    import torch

    from paper_2408_14267_amd import fqt
    from paper_2408_14267_amd.workloads import WORKLOADS, LayerShape
    dev = torch.device("cuda:0")
    st = torch.cuda.current_stream()
    torch.manual_seed(0)

    def timed(fn, k):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(st)
        for _ in range(k):
            fn()
        e1.record(st)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / k

    if name == "table5":
        # The paper's Table 5 sizes (m, k, n): a gradient of m columns over a k-deep contraction
        # times k x n signs (reading of its unlabeled rows: m is the pruned side).  Average
        # 1-bit: b = 4 codes of the m / 4 columns top-k keeps; 1-bit: b = 1 codes of all m, no
        # pruning.  Both run the dW product entry; only the product is timed.  Then the same
        # shapes scaled by 8 in every dimension, where the product is no longer latency-bound.
        paper = {(512, 512, 512): (8.40, 8.01), (512, 512, 1024): (15.92, 14.54),
                 (1024, 512, 512): (16.61, 15.91), (1024, 512, 1024): (31.03, 29.79),
                 (2048, 512, 512): (32.22, 29.92), (2048, 512, 1024): (61.33, 59.94)}
        scaled = {(8 * m, 8 * k, 8 * n): (None, None) for (m, k, n) in paper}
        for (m, k, n), (p_avg, p_one) in list(paper.items()) + list(scaled.items()):
            L = LayerShape(name="mm", kind="linear", N=k, C=n, D=m)
            desc = fqt.layer_desc(L)
            dY = _gen(torch, (k, m), torch.float32, dev)
            X = _gen(torch, (k, n), torch.float32, dev)
            xs = torch.empty(((k + 63) // 64) * n, dtype=torch.int64, device=dev)
            fqt.fqt_pack_input_signs(desc, X, xs, st)
            dW = torch.empty((m, n), dtype=torch.float32, device=dev)
            out = {"suite": name, "m_k_n": [m, k, n]}
            for tag, cfg in (("avg1bit", fqt.quant_cfg(4, fqt.FQT_AGP_TOPK, 0, 0, 0)),
                             ("1bit", fqt.quant_cfg(1, fqt.FQT_AGP_OFF, 0, 0, 0))):
                q = fqt.QGrad(desc, cfg, device=dev)
                qws = fqt.workspace(desc, cfg, fqt.FQT_WS_QUANTIZE, device=dev)
                dws = fqt.workspace(desc, cfg, fqt.FQT_WS_GEMM_DW, device=dev)
                fqt.fqt_agp_scq_quantize(desc, cfg, dY, q, qws, st)
                gd = lambda: fqt.fqt_binary_gemm_dw(desc, cfg, q, xs, dW, dws, None, st)
                for _ in range(3):
                    gd()
                out[tag + "_ms"] = round(timed(gd, 50), 5)
                out[tag + "_kept"] = int(q.pcq_count.item())
            out["ratio"] = round(out["avg1bit_ms"] / out["1bit_ms"], 3)
            if p_avg is not None:
                out["paper_hygon_ms"] = [p_avg, p_one]
                out["paper_ratio"] = round(p_avg / p_one, 3)
            else:
                out["sizes"] = "the paper's sizes x 8 in each dimension"
            print(json.dumps(out), flush=True)
            del dY, X, xs, dW, q, qws, dws
            torch.cuda.empty_cache()
        return

    if name == "forward":
        for wname in (WORKLOAD, "resnet18_32px", "vgg16_224_bf16"):
            wl = WORKLOADS[wname]
            tdt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
            tot_ms, tot_ops = 0.0, 0.0
            for li, L in enumerate(wl.layers):
                X = _gen(torch, L.x_shape, tdt, dev)
                W = _gen(torch, L.w_shape, torch.float32, dev)
                G = _gen(torch, (L.D,), torch.float32, dev)
                Y = torch.empty(L.dy_shape, dtype=tdt, device=dev)
                dt = fqt.FQT_BF16 if tdt == torch.bfloat16 else fqt.FQT_F32
                desc = fqt.layer_desc(L, dt, dt, fqt.FQT_F32, dt)
                ws = fqt.workspace(desc, None, fqt.FQT_WS_FORWARD, device=dev)
                step = lambda: fqt.fqt_binary_forward(desc, X, W, G, Y, None, ws, st)
                for _ in range(3):
                    step()
                ms = timed(step, reps)
                ops = 2.0 * L.binary_macs()
                tot_ms += ms
                tot_ops += ops
                print(json.dumps({"suite": name, "workload": wname, "layer": li, "name": L.name,
                                  "ms": round(ms, 4), "binary_TOPS": round(ops / ms / 1e9, 1),
                                  "mfma_frac": round(ops / ms / 1e9 / MFMA_I8_PEAK_TOPS, 4)}),
                      flush=True)
                del X, W, G, Y, ws
                torch.cuda.empty_cache()
            print(json.dumps({"suite": name, "workload": wname, "total_ms": round(tot_ms, 3),
                              "binary_TOPS": round(tot_ops / tot_ms / 1e9, 1)}), flush=True)
        return

    if name == "gemm_sweep":
        from paper_2408_14267_amd.workloads import gemm_sweep_points
        for M, _, K in gemm_sweep_points():
            # dW of a linear layer with batch K, in = out = M: an M x M x K binary GEMM of
            # 1-bit codes (b = 1, no pruning) against packed signs.
            L = LayerShape(name="gemm", kind="linear", N=K, C=M, D=M)
            desc = fqt.layer_desc(L)
            cfg = fqt.quant_cfg(1, fqt.FQT_AGP_OFF, 0, 0, 0)
            dY = _gen(torch, (K, M), torch.float32, dev)
            X = _gen(torch, (K, M), torch.float32, dev)
            q = fqt.QGrad(desc, cfg, device=dev)
            qws = fqt.workspace(desc, cfg, fqt.FQT_WS_QUANTIZE, device=dev)
            dws = fqt.workspace(desc, cfg, fqt.FQT_WS_GEMM_DW, device=dev)
            xs = torch.empty(((K + 63) // 64) * M, dtype=torch.int64, device=dev)
            dW = torch.empty((M, M), dtype=torch.float32, device=dev)
            qz = lambda: fqt.fqt_agp_scq_quantize(desc, cfg, dY, q, qws, st)
            px = lambda: fqt.fqt_pack_input_signs(desc, X, xs, st)
            gd = lambda: fqt.fqt_binary_gemm_dw(desc, cfg, q, xs, dW, dws, None, st)
            for f in (qz, px, gd):
                f()
            k = 3 if M * M * K > 2 ** 36 else reps
            tq, tp, tg = timed(qz, k), timed(px, k), timed(gd, k)
            ops = 2.0 * M * M * K
            # quantize: dY read twice (statistics, codes) + 1-byte codes and b-bit planes of
            # both encodings written
            qbytes = K * M * 4 * 2 + 2 * K * M + 2 * K * M / 8
            print(json.dumps({"suite": name, "gemm_MxNxK": [M, M, K],
                              "gemm_dw_ms": round(tg, 4), "int8_TOPS": round(ops / tg / 1e9, 1),
                              "mfma_frac": round(ops / tg / 1e9 / MFMA_I8_PEAK_TOPS, 4),
                              "quantize_ms": round(tq, 4),
                              "quantize_GBps": round(qbytes / tq / 1e6, 1),
                              "pack_x_ms": round(tp, 4)}), flush=True)
            del dY, X, q, qws, dws, xs, dW
            torch.cuda.empty_cache()
        return

    wl = WORKLOADS[name]
    tdt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    tot_ms, tot_ops = 0.0, 0.0
    for li, L in enumerate(wl.layers):
        X = _gen(torch, L.x_shape, tdt, dev)
        W = _gen(torch, L.w_shape, torch.float32, dev)
        nd = len(L.dy_shape)
        r = wl.recipe
        if r.kind == "sample_lognormal":
            sc = torch.exp(r.sigma * torch.randn((L.N,) + (1,) * (nd - 1), device=dev))
            dY = _gen(torch, L.dy_shape, tdt, dev, sc)
        elif r.kind == "channel_lognormal":
            sc = torch.exp(r.sigma * torch.randn((1, L.D) + (1,) * (nd - 2), device=dev))
            dY = _gen(torch, L.dy_shape, tdt, dev, sc)
        else:
            dY = torch.distributions.StudentT(r.df).sample(L.dy_shape).to(dev).to(tdt)
        dX, dW = torch.empty_like(X), torch.empty_like(W)
        if tdt == torch.bfloat16:
            desc = fqt.layer_desc(L, fqt.FQT_BF16, fqt.FQT_BF16, fqt.FQT_F32, fqt.FQT_BF16)
        else:
            desc = fqt.layer_desc(L)
        cfg = fqt.quant_cfg(wl.bits, wl.agp_mode, wl.philox_seed, 0, li)
        ws = fqt.workspace(desc, cfg, device=dev)
        step = lambda: fqt.fqt_layer_backward(desc, cfg, X, W, dY, dX, dW, ws, st)
        for _ in range(3):
            step()
        ms = timed(step, reps)
        ops = 4.0 * L.binary_macs()
        es = 2 if tdt == torch.bfloat16 else 4
        # each tensor crossing HBM once: dY, X, W read; dX, dW written
        mbytes = (L.N * L.D * L.Ho * L.Wo + 2 * L.N * L.C * L.H * L.W) * es + 2 * L.D * L.C * L.kh * L.kw * 4
        tot_ms += ms
        tot_ops += ops
        print(json.dumps({"suite": name, "layer": li, "name": L.name, "ms": round(ms, 4),
                          "binary_TOPS": round(ops / ms / 1e9, 1),
                          "min_bytes_MB": round(mbytes / 1e6, 2),
                          "GBps_of_min_bytes": round(mbytes / ms / 1e6, 1)}), flush=True)
        del X, W, dY, dX, dW, ws
        torch.cuda.empty_cache()
    print(json.dumps({"suite": name, "total_ms": round(tot_ms, 3),
                      "binary_TOPS": round(tot_ops / tot_ms / 1e9, 1)}), flush=True)


def main():
    args = parse()
    if args.suite:
        if args.gpus != 1:
            sys.exit("the suites run on one GPU")
        suite(args.suite)
        return
    if args.gpus != 1:
        print(json.dumps({"error": "this benchmark runs on one GPU only; the layer backward "
                                   "would shard by data parallelism with one dW all-reduce, "
                                   "which is not implemented", "n_gpus": args.gpus}))
        sys.exit(2)

    import torch

    from paper_2408_14267_amd import fqt
    from paper_2408_14267_amd.workloads import WORKLOADS, draw_layer

    wl = WORKLOADS[WORKLOAD]
    layer = wl.layers[0]
    dev = torch.device("cuda:0")
    if args.calib_copy_mib:
        src = torch.ones(args.calib_copy_mib << 18, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
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

    def graph_of(fn, reps):
        """A HIP graph of `reps` back-to-back calls of fn(stream), captured on a side stream."""
        g = torch.cuda.CUDAGraph()
        side = torch.cuda.Stream()
        side.wait_stream(stream)
        with torch.cuda.stream(side):
            fn(side)
            torch.cuda.synchronize()
            with torch.cuda.graph(g, stream=side):
                for _ in range(reps):
                    fn(side)
        torch.cuda.synchronize()
        return g

    ms_graph = None
    if not args.no_graph:
        g = graph_of(lambda st: fqt.fqt_layer_backward(desc, cfg, X, W, dY, dX, dW, ws, st), 1)
        for _ in range(args.warmup):
            g.replay()
        ms_graph = timed(g.replay, args.steps)
    # The step is reported in the faster of the two launch modes (same work either way).
    ms = ms_eager if ms_graph is None else min(ms_eager, ms_graph)

    # Single-kernel entry points, each timed as a graph of REPS back-to-back launches replayed
    # on `stream` between two HIP events (eager launches of a few-microsecond kernel would
    # time the host instead).
    q = fqt.QGrad(desc, cfg, device=dev)
    qws = fqt.workspace(desc, cfg, fqt.FQT_WS_QUANTIZE, device=dev)
    dws = fqt.workspace(desc, cfg, fqt.FQT_WS_GEMM_DW, device=dev)
    K = layer.C * layer.kh * layer.kw
    P = layer.Ho * layer.Wo
    R = layer.N * P
    Wd, Wr = (layer.D + 63) // 64, (R + 63) // 64
    xs = torch.empty(Wr * K, dtype=torch.int64, device=dev)
    wsb = torch.empty(K, 64 * Wd, dtype=torch.int8, device=dev)
    wls = torch.empty(K, dtype=torch.int32, device=dev)
    entries = {
        "quantize": lambda st: fqt.fqt_agp_scq_quantize(desc, cfg, dY, q, qws, st),
        "pack_x": lambda st: fqt.fqt_pack_input_signs(desc, X, xs, st),
        "pack_w": lambda st: fqt.fqt_pack_weight_signs(desc, W, wsb, wls, st),
        "gemm_dw": lambda st: fqt.fqt_binary_gemm_dw(desc, cfg, q, xs, dW, dws, None, st),
        "gemm_dx": lambda st: fqt.fqt_binary_gemm_dx(desc, cfg, q, wsb, wls, dX, None, st),
    }
    REPS = 20
    per = {}
    for name, fn in entries.items():
        if args.no_graph:
            for _ in range(args.warmup):
                fn(stream)
            per[name] = timed(lambda: fn(stream), args.steps)
            continue
        gk = graph_of(fn, REPS)
        for _ in range(max(1, args.warmup // REPS)):
            gk.replay()
        per[name] = timed(gk.replay, max(1, args.steps // REPS)) / REPS
    ks, kc = int(q.psq_count.item()), int(q.pcq_count.item())
    b = wl.bits
    # Algorithmic bytes (each tensor crosses HBM once; codes at b bits, signs at 1 bit) and
    # int8 MFMA ops (2 * M * N * K over the kept rows) of each single-kernel entry.
    work = {
        "pack_x": (X.numel() * 4 + K * Wr * 8, 0),
        "pack_w": (W.numel() * 4 + K * Wd * 8, 0),
        "gemm_dw": (kc * R * b // 8 + K * Wr * 8 + dW.numel() * 4, 2 * kc * K * R),
        "gemm_dx": (ks * P * layer.D * b // 8 + K * Wd * 8 + dX.numel() * 4,
                    2 * ks * layer.H * layer.W * layer.C * K * layer.D // layer.C),
    }
    # The roofline is taken on the longest entry point that launches a single kernel (the
    # dW entry launches two: split partials and their sum; the quantizer three).
    dom = max(("gemm_dx", "pack_x", "pack_w"), key=lambda k: per[k])
    nbytes, nops = work[dom]
    t_s = per[dom] * 1e-3
    if nbytes / (HBM_PEAK_GBS * 1e9) >= nops / (MFMA_I8_PEAK_TOPS * 1e12):
        roofline = {"bound": "hbm", "achieved": nbytes / t_s / 1e9, "peak": HBM_PEAK_GBS,
                    "unit": "GB/s", "frac": nbytes / t_s / 1e9 / HBM_PEAK_GBS}
    else:
        roofline = {"bound": "mfma", "achieved": nops / t_s / 1e12, "peak": MFMA_I8_PEAK_TOPS,
                    "unit": "TOPS", "frac": nops / t_s / 1e12 / MFMA_I8_PEAK_TOPS}
    roofline.update({"traffic": measured_traffic(dom), "kernel": dom, "kernel_ms": per[dom],
                     "algorithmic_bytes": nbytes, "int8_ops": nops,
                     "kept_samples": ks, "kept_channels": kc})

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
        "dtype": "u1/i8->i32",
        "data": "synthetic",
        "config": {"workload": WORKLOAD, "layer": "conv3x3 256->256, 8x8, stride 1, pad 1",
                   "batch": layer.N, "bits": wl.bits, "agp": "bernoulli", "inputs": "f32",
                   "accumulate": "i32",
                   "timed_as": "hip_graph" if ms_graph is not None and ms_graph <= ms_eager else "eager",
                   "ms_per_step_eager": ms_eager, "ms_per_step_graph": ms_graph,
                   "per_kernel_ms": per, "binary_ops_per_step": ops_per_step},
        "roofline": roofline,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out))


if __name__ == "__main__":
    main()
