"""Benchmark of the 1-bit FQT layer backward on one MI355X.

Workload: VGG-16 CIFAR-shaped 3x3 convolution 256 -> 256 on 8x8 maps, batch 128,
fp32 X / W / dY (dY per-sample lognormal(0, 2) scale with 13 of 128 samples x100),
AGP Bernoulli keeping 1/4 of the groups (b = 4), Philox seed 0.  A step is one
fqt_layer_backward: group statistics, AGP selection, SR + code packing, sign packing
of X (bit-im2col) and W, and both binary products with rescale.

Prints one JSON line: throughput in binary TOPS (2 x D*C*k*k*N*Ho*Wo binary
multiply-accumulates per product, both products, per step time); the roofline of the
step's dominant kernel (the products launch, timed alone with HIP events on its stream)
and of the whole step; the linear 32x256x128 layer, and the ResNet-18 (32 px, batch 128)
and VGG-16 (224 px, batch 64, bf16) backward passes over all their layers, eager and as
one HIP graph; a cold-cache step time; and the CPU oracle timed on a bounded sample on
the host, on one thread and on all of the process's cores.
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
MFMA_FP4_PEAK_TOPS = 10100.0   # MI355X dense fp4 MFMA
# VALU popcount: 256 CUs x 64 lanes x 2.4 GHz lane-ops; AND + popcount-accumulate of a 64-bit
# word pair is 4 lane-ops for 64 binary multiply-accumulates (128 binary ops).
POPC_PEAK_TOPS = 256 * 64 * 2.4e9 / 4 * 128 / 1e12
GRAPH_STEPS = 10               # layer steps per graph in the graph-mode timing
SCRUB_BYTES = 1 << 30          # cold-cache runs overwrite this much (the last-level cache is 256 MB)

# HBM traffic per launch of the products kernel from rocprofv3 counter runs of this benchmark
# (FETCH_SIZE and WRITE_SIZE in KiB per dispatch, one run each), scaled by what the same
# counters read for a 256 MiB device copy in those runs.  Reported only while the kernel
# sources are byte-identical to the ones they were measured on (TRAFFIC_DIGEST: sha256 over
# the names and contents of every file in csrc/).
FETCH_SCALE = 262144.0 / 131086.6
WRITE_SCALE = 262144.0 / 262144.0
TRAFFIC_DIGEST = "61a4f7869ca7d7426b35ca8bf86bc4293fc04e8f6ce585ac75fd8e5c4a4ff2ee"
TRAFFIC = {       # kernel: (FETCH_SIZE KiB, WRITE_SIZE KiB) per launch
    "products": (6194.3, 10496.0),
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
    p.add_argument("--cpu-seconds", type=float, default=8.0,
                   help="bound on each CPU oracle leg (seconds of work)")
    p.add_argument("--no-graph", action="store_true", help="time eager launches only")
    p.add_argument("--no-networks", action="store_true",
                   help="skip the ResNet-18 and VGG-16 whole-network totals")
    p.add_argument("--cold", action="store_true",
                   help="report the cold-cache step time as ms_per_step (1 GiB overwritten "
                        "before every timed step) instead of the warm one")
    p.add_argument("--suite", choices=("resnet18_32px", "vgg16_224_bf16", "gemm_sweep", "forward",
                                       "table5", "train", "variance", "baselines", "engines"),
                   help="instead of the benchmark line: per-layer times of a whole network's "
                        "layer backwards, the dW binary GEMM sweep, the binary forward of "
                        "the VGG CIFAR conv layer and of every ResNet-18 / VGG-16 layer, or "
                        "average-1-bit against 1-bit products at the sizes of the paper's "
                        "Table 5 (one JSON line each)")
    p.add_argument("--calib-copy-mib", type=int, default=0,
                   help="first run a plain device copy of this many MiB (three times), so that "
                        "a counter run can scale FETCH_SIZE / WRITE_SIZE by a known byte count")
    return p.parse_args()


def cpu_legs(x, w, dy, layer, wl, ops_per_step, budget_s):
    """The oracle, as it stands, on the host: a full layer backward repeated until about
    `budget_s` seconds of work have been done (at least once), first with every thread pool
    held to one thread (the paper times one core), then with the pools at the process's
    cores.  Returns (one-thread leg, all-cores leg)."""
    from threadpoolctl import threadpool_info, threadpool_limits

    from oracle import fqt as ofqt
    cores = len(os.sched_getaffinity(0))

    def run(threads):
        with threadpool_limits(limits=threads):
            used = max([1] + [int(i.get("num_threads", 1)) for i in threadpool_info()])
            reps, t0 = 0, time.perf_counter()
            while True:
                ofqt.layer_backward(x, w, dy, wl.bits, wl.agp_mode, seed=wl.philox_seed,
                                    stride=layer.stride, pad=layer.pad)
                reps += 1
                el = time.perf_counter() - t0
                if el >= budget_s:
                    break
        return {"value": ops_per_step * reps / el / 1e12, "unit": "TOPS", "cores": used,
                "kind": "oracle", "ms_per_step": el / reps * 1e3,
                "sample": f"{reps} full layer backward(s) of {WORKLOAD} in {el:.1f} s "
                          f"({el / reps * 1e3:.0f} ms each; numpy, thread pools at {used} "
                          f"of the process's {cores} cores)"}
    return run(1), run(cores)


def _gen(torch, shape, dtype, dev, scale=None):
    x = torch.randn(shape, device=dev, dtype=torch.float32)
    if scale is not None:
        x *= scale
    return x.to(dtype)


def _dequantized(torch, q, N, D, P):
    """(PSQ estimate, PCQ estimate) of dY as float64 [N][D][P], from the codes, kept lists,
    scales and offsets of a quantized gradient (the estimate g_hat = S q + Z' of the kept
    groups, 0 elsewhere)."""
    R = N * P
    Wd, Wr = (D + 63) // 64, (R + 63) // 64
    out = []
    for side in ("psq", "pcq"):
        count = int(getattr(q, side + "_count").item())
        kept = getattr(q, side + "_kept")[:count].long()
        S = getattr(q, side + "_scale").double()[kept]
        Z = getattr(q, side + "_offset").double()[kept]
        g = torch.zeros((N, D, P), dtype=torch.float64, device=q.psq_codes.device)
        if side == "psq":
            codes = q.psq_codes.view(2 * Wd, R, 32).permute(1, 0, 2).reshape(R, 64 * Wd)[:, :D]
            rows = codes[:count * P].double().view(count, P, D).permute(0, 2, 1)
            g[kept] = S[:, None, None] * rows + Z[:, None, None]
        else:
            codes = q.pcq_codes.view(2 * Wr, D, 32).permute(1, 0, 2).reshape(D, 64 * Wr)[:, :R]
            rows = codes[:count].double().view(count, N, P).permute(1, 0, 2)
            g[:, kept] = S[None, :, None] * rows + Z[None, :, None]
        out.append(g)
    return out


def _draw_dy(torch, L, recipe, dtype, dev):
    nd = len(L.dy_shape)
    if recipe.kind == "sample_lognormal":
        sc = torch.exp(recipe.sigma * torch.randn((L.N,) + (1,) * (nd - 1), device=dev))
        return _gen(torch, L.dy_shape, dtype, dev, sc)
    if recipe.kind == "channel_lognormal":
        sc = torch.exp(recipe.sigma * torch.randn((1, L.D) + (1,) * (nd - 2), device=dev))
        return _gen(torch, L.dy_shape, dtype, dev, sc)
    return torch.distributions.StudentT(recipe.df).sample(L.dy_shape).to(dev).to(dtype)


def _timed(torch, stream, fn, k):
    """Mean ms of k calls of fn between two HIP events recorded on `stream`."""
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(k):
        fn()
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / k


def _graph_of(torch, stream, fn, reps):
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


def network_layers(name, dev, stream, reps=10, graph=True, per_layer=None, bits=None,
                   agp_mode=None):
    """Every layer backward of a network (inputs drawn on the GPU with the workload's recipe
    distributions, one workspace shared by all layers): per-layer eager ms, the eager total,
    and one HIP graph of the whole network's layer calls replayed (ms per pass)."""
    import torch

    from paper_2408_14267_amd import fqt
    from paper_2408_14267_amd.workloads import WORKLOADS
    torch.manual_seed(0)
    wl = WORKLOADS[name]
    tdt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    calls, ws_bytes, rows = [], 0, []
    for li, L in enumerate(wl.layers):
        X = _gen(torch, L.x_shape, tdt, dev)
        W = _gen(torch, L.w_shape, torch.float32, dev)
        dY = _draw_dy(torch, L, wl.recipe, tdt, dev).contiguous()
        dX, dW = torch.empty_like(X), torch.empty_like(W)
        if tdt == torch.bfloat16:
            desc = fqt.layer_desc(L, fqt.FQT_BF16, fqt.FQT_BF16, fqt.FQT_F32, fqt.FQT_BF16)
        else:
            desc = fqt.layer_desc(L)
        cfg = fqt.quant_cfg(wl.bits if bits is None else bits,
                            wl.agp_mode if agp_mode is None else agp_mode, wl.philox_seed, 0, li)
        ws_bytes = max(ws_bytes, fqt.fqt_workspace_size(desc, cfg))
        calls.append((L, desc, cfg, X, W, dY, dX, dW))
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    fqt.fqt_workspace_init(ws, stream)

    def layer_fn(c, st):
        L, desc, cfg, X, W, dY, dX, dW = c
        fqt.fqt_layer_backward(desc, cfg, X, W, dY, dX, dW, ws, st)

    total_eager, ops = 0.0, 0.0
    es = 2 if tdt == torch.bfloat16 else 4
    for li, c in enumerate(calls):
        L = c[0]
        step = lambda: layer_fn(c, stream)
        for _ in range(3):
            step()
        ms = _timed(torch, stream, step, reps)
        total_eager += ms
        ops += 4.0 * L.binary_macs()
        mbytes = (L.N * L.D * L.Ho * L.Wo + 2 * L.N * L.C * L.H * L.W) * es + \
            2 * L.D * L.C * L.kh * L.kw * 4
        rows.append({"layer": li, "name": L.name, "ms": round(ms, 4),
                     "binary_TOPS": round(4.0 * L.binary_macs() / ms / 1e9, 1),
                     "min_bytes_MB": round(mbytes / 1e6, 2),
                     "GBps_of_min_bytes": round(mbytes / ms / 1e6, 1)})
        if per_layer:
            per_layer({"suite": name, **rows[-1]})
    out = {"layers": len(calls), "ms_eager": round(total_eager, 4),
           "binary_TOPS_eager": round(ops / total_eager / 1e9, 1)}
    if graph:
        g = _graph_of(torch, stream, lambda st: [layer_fn(c, st) for c in calls], 1)
        for _ in range(3):
            g.replay()
        ms_g = _timed(torch, stream, g.replay, reps)
        out.update({"ms_graph": round(ms_g, 4), "binary_TOPS_graph": round(ops / ms_g / 1e9, 1)})
    out["min_bytes_MB"] = round(sum(r["min_bytes_MB"] for r in rows), 1)
    if name.startswith("resnet18"):
        # The layers the paper quantizes: all but the stem conv, the fc and the 1x1 shortcuts.
        sub = [r for r in rows if r["name"] not in ("conv1", "fc") and not r["name"].endswith(".down")]
        out["quantized_subset"] = {"layers": len(sub),
                                   "ms_eager": round(sum(r["ms"] for r in sub), 4)}
    del calls, ws
    torch.cuda.empty_cache()
    return out, rows


def suite(name, reps=10):
    """One JSON line per layer / point: a whole network's layer backwards (per-layer eager
    times, then the totals eager and as one graph), the dW binary GEMM sweep, the binary
    forward, or the Table 5 analogue."""
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

    if name == "train":
        # A Table 3 analogue: one training step (forward, cross-entropy, backward, Adam) of
        # VGG-16 and ResNet-18 at 32 x 32 (batch 128) and 224 x 224 (batch 64), random data:
        # the binary network under 1-bit FQT (b = 4, AGP Bernoulli) against the same network
        # in float32 and in bf16 autocast on the same GPU.
        from paper_2408_14267_amd import train
        for net, res, nb in (("vgg16", 32, 128), ("resnet18", 32, 128), ("vgg16", 224, 64),
                             ("resnet18", 224, 64)):
            out = {"suite": name, "net": net, "res": res, "batch": nb}
            for mode in ("binary_fqt", "fp32", "bf16_autocast"):
                torch.manual_seed(0)
                binary = mode == "binary_fqt"
                classes = 10 if res == 32 else 1000
                model = (train.VGG16(classes, res, binary=binary, bits=4) if net == "vgg16"
                         else train.ResNet18(classes, binary=binary, bits=4)).to(dev)
                opt = torch.optim.Adam(model.parameters(), lr=1e-3)
                x = torch.randn(nb, 3, res, res, device=dev)
                y = torch.randint(0, classes, (nb,), device=dev)
                ac = torch.bfloat16 if mode == "bf16_autocast" else None
                stepf = lambda: train.train_step(model, opt, x, y, ac)
                for _ in range(3):
                    stepf()
                out[mode + "_ms"] = round(timed(stepf, reps), 4)
                del model, opt
                torch.cuda.empty_cache()
            out["speedup_vs_fp32"] = round(out["fp32_ms"] / out["binary_fqt_ms"], 3)
            out["speedup_vs_bf16"] = round(out["bf16_autocast_ms"] / out["binary_fqt_ms"], 3)
            print(json.dumps(out), flush=True)
        return

    if name == "variance":
        # Quantizer variance (Section 4.2; the paper's per-layer variance figure for
        # ResNet-18): E sum (g_hat - dY)^2 of the estimate that feeds each product, estimated
        # from the GPU quantizer over 32 Philox steps, for 1-bit per-group quantization
        # without AGP (the PSQ baseline) and for AGP + b-bit codes, b = 2, 4, 8.  Relative to
        # sum dY^2, and as a fraction of the 1-bit baseline.
        from paper_2408_14267_amd.workloads import WORKLOADS as WL
        steps = 32
        points = [("vgg_cifar_conv3x3_256", 0, WL["vgg_cifar_conv3x3_256"].layers[0])] + \
                 [("resnet18_32px", i, L) for i, L in enumerate(WL["resnet18_32px"].layers)]
        for wname, li, L in points:
            wl = WL[wname]
            dY = _draw_dy(torch, L, wl.recipe, torch.float32, dev).contiguous()
            N, D, P = L.N, L.D, L.Ho * L.Wo
            x = dY.double().view(N, D, P)
            norm = float((x * x).sum())
            desc = fqt.layer_desc(L)
            row = {"suite": name, "workload": wname, "layer": li, "name": L.name,
                   "sum_dY2": norm, "steps": steps}
            for tag, bits, mode in (("psq1_no_agp", 1, fqt.FQT_AGP_OFF),
                                    ("agp_b2", 2, fqt.FQT_AGP_BERNOULLI),
                                    ("agp_b4", 4, fqt.FQT_AGP_BERNOULLI),
                                    ("agp_b8", 8, fqt.FQT_AGP_BERNOULLI)):
                ts, tc = 0.0, 0.0
                for step in range(steps):
                    cfg = fqt.quant_cfg(bits, mode, 0, step, li)
                    q = fqt.QGrad(desc, cfg, device=dev)
                    fqt.fqt_agp_scq_quantize(desc, cfg, dY, q,
                                             fqt.workspace(desc, cfg, fqt.FQT_WS_QUANTIZE,
                                                           device=dev), st)
                    gs, gc = _dequantized(torch, q, N, D, P)
                    ts += float(((gs - x) ** 2).sum())
                    tc += float(((gc - x) ** 2).sum())
                row[tag] = {"psq_rel_var": ts / steps / norm, "pcq_rel_var": tc / steps / norm}
            for tag in ("agp_b2", "agp_b4", "agp_b8"):
                row[tag]["psq_vs_1bit"] = row[tag]["psq_rel_var"] / row["psq1_no_agp"]["psq_rel_var"]
                row[tag]["pcq_vs_1bit"] = row[tag]["pcq_rel_var"] / row["psq1_no_agp"]["pcq_rel_var"]
            print(json.dumps(row), flush=True)
            del dY, x
            torch.cuda.empty_cache()
        return

    if name == "baselines":
        # Baseline quantizers on the same kernels (the paper's Table 1 / Table 3 rows), on the
        # 256 -> 256 conv (8 x 8, batch 128) and the ResNet-18 network: ours (AGP, b = 4),
        # 1-bit per-group codes without AGP, 8-bit SCQ without AGP; and 8-bit PSQ for both
        # products, where dW cannot use the integer kernels (its per-sample scale varies along
        # the contraction, Section 5.3): the dX product on the kernels, dW as a float32
        # product of the dequantized PSQ gradient with sign(unfold(X)) (torch, a comparison
        # system only).
        from paper_2408_14267_amd.workloads import WORKLOADS as WL
        variants = (("ours_agp_b4", 4, fqt.FQT_AGP_BERNOULLI), ("scq1_no_agp", 1, fqt.FQT_AGP_OFF),
                    ("scq8_no_agp", 8, fqt.FQT_AGP_OFF))
        wl = WL["vgg_cifar_conv3x3_256"]
        L = wl.layers[0]
        X = _gen(torch, L.x_shape, torch.float32, dev)
        W = _gen(torch, L.w_shape, torch.float32, dev)
        dY = _draw_dy(torch, L, wl.recipe, torch.float32, dev).contiguous()
        dX, dW = torch.empty_like(X), torch.empty_like(W)
        desc = fqt.layer_desc(L)
        row = {"suite": name, "workload": wl.name}
        for tag, bits, mode in variants:
            cfg = fqt.quant_cfg(bits, mode, 0, 0, 0)
            ws = fqt.workspace(desc, cfg, device=dev)
            f = lambda: fqt.fqt_layer_backward(desc, cfg, X, W, dY, dX, dW, ws, st)
            for _ in range(5):
                f()
            row[tag + "_ms"] = round(timed(f, 50), 5)
        # 8-bit PSQ for both products.
        cfg = fqt.quant_cfg(8, fqt.FQT_AGP_OFF, 0, 0, 0)
        q = fqt.QGrad(desc, cfg, device=dev)
        qws = fqt.workspace(desc, cfg, fqt.FQT_WS_QUANTIZE, device=dev)
        K, P = L.C * L.kh * L.kw, L.Ho * L.Wo
        Wd = (L.D + 63) // 64
        wsb = torch.empty(K, 64 * Wd, dtype=torch.int8, device=dev)
        wls = torch.empty(K, dtype=torch.int32, device=dev)

        def psq8_both():
            fqt.fqt_agp_scq_quantize(desc, cfg, dY, q, qws, st)
            fqt.fqt_pack_weight_signs(desc, W, wsb, wls, st)
            fqt.fqt_binary_gemm_dx(desc, cfg, q, wsb, wls, dX, None, st)
            gs = _dequantized(torch, q, L.N, L.D, P)[0].float()             # [N][D][P]
            sx = torch.nn.functional.unfold(X, (L.kh, L.kw), padding=(L.ph, L.pw),
                                            stride=(L.sh, L.sw))             # [N][K][P]
            sx = torch.where(sx > 0, 1.0, -1.0)
            dW.view(L.D, K).copy_(gs.permute(1, 0, 2).reshape(L.D, -1)
                                  @ sx.permute(1, 0, 2).reshape(K, -1).t())
        for _ in range(5):
            psq8_both()
        row["psq8_both_products_ms"] = round(timed(psq8_both, 50), 5)
        print(json.dumps(row), flush=True)
        del X, W, dY, dX, dW
        torch.cuda.empty_cache()
        # The ResNet-18 network, per variant (eager totals).
        for tag, bits, mode in variants:
            wl18 = WL["resnet18_32px"]
            out, _ = network_layers("resnet18_32px", dev, st, reps=10, graph=False,
                                    bits=bits, agp_mode=mode)
            print(json.dumps({"suite": name, "workload": "resnet18_32px", "variant": tag,
                              "ms_eager": out["ms_eager"]}), flush=True)
        return

    if name == "engines":
        # The dW product on the three engines (Section 5.2 decomposition; Appendix C binary
        # multiplication): int8 MFMA over the byte codes (the library's), VALU popcount over
        # the bit planes (the paper's), and gfx950's fp4 MFMA over the planes expanded to
        # e2m1.  Each against its own peak: int8 ops 2 * kept * K * R; popcount and fp4 issue
        # one pass per plane, 2 * b * kept * K * R.  The fp4 time includes its expansion
        # launches; the expansion-free product time is reported beside it.
        from paper_2408_14267_amd.workloads import WORKLOADS as WL, gemm_sweep_points
        pts = [("vgg_cifar_conv3x3_256", WL["vgg_cifar_conv3x3_256"].layers[0], 4,
                fqt.FQT_AGP_BERNOULLI)]
        pts += [(f"gemm_{M}x{M}x{K}", LayerShape(name="g", kind="linear", N=K, C=M, D=M), 1,
                 fqt.FQT_AGP_OFF) for M, _, K in gemm_sweep_points() if M <= 8192]
        for wname, L, bits, mode in pts:
            desc = fqt.layer_desc(L)
            cfg = fqt.quant_cfg(bits, mode, 0, 0, 0)
            X = _gen(torch, L.x_shape, torch.float32, dev)
            dY = _gen(torch, L.dy_shape, torch.float32, dev).contiguous()
            K, P = L.C * L.kh * L.kw, L.Ho * L.Wo
            R = L.N * P
            Wr = (R + 63) // 64
            q = fqt.QGrad(desc, cfg, device=dev)
            fqt.fqt_agp_scq_quantize(desc, cfg, dY, q,
                                     fqt.workspace(desc, cfg, fqt.FQT_WS_QUANTIZE, device=dev), st)
            xwm = torch.empty(Wr * K, dtype=torch.int64, device=dev)
            fqt.fqt_pack_input_signs(desc, X, xwm, st)
            xb = torch.empty(K * Wr, dtype=torch.int64, device=dev)
            xs = torch.empty(K, dtype=torch.int32, device=dev)
            if L.kind == "linear":
                fqt.fqt_pack_bits(X, fqt.FQT_F32, L.N, L.C, L.C, fqt.FQT_PACK_ALONG_ROWS, None, xb,
                                  xs, st)
            else:
                fqt.fqt_pack_bits(X, fqt.FQT_F32, 0, 0, 0, fqt.FQT_PACK_IM2COL, desc, xb, xs, st)
            dW = torch.empty((L.D, K), device=dev)
            kept = int(q.pcq_count.item())
            macs = kept * K * R
            reps = 3 if macs > 2 ** 38 else 20
            row = {"suite": name, "workload": wname, "bits": bits, "kept_channels": kept,
                   "K": K, "R": R}
            dws = fqt.workspace(desc, cfg, fqt.FQT_WS_GEMM_DW, device=dev)
            f8 = lambda: fqt.fqt_binary_gemm_dw(desc, cfg, q, xwm, dW, dws, None, st)
            f8()
            t8 = timed(f8, reps)
            row["int8"] = {"ms": round(t8, 5), "TOPS": round(2 * macs / t8 / 1e9, 1),
                           "frac_of_peak": round(2 * macs / t8 / 1e9 / MFMA_I8_PEAK_TOPS, 4)}
            for tag, eng, which, peak in (("popcount", fqt.FQT_ENGINE_POPCOUNT,
                                           fqt.FQT_WS_DW_POPCOUNT, POPC_PEAK_TOPS),
                                          ("fp4", fqt.FQT_ENGINE_FP4, fqt.FQT_WS_DW_FP4,
                                           MFMA_FP4_PEAK_TOPS)):
                if tag == "fp4" and bits > 4:
                    continue
                ws_e = fqt.workspace(desc, cfg, which, device=dev)
                fe = lambda: fqt.fqt_binary_gemm_dw_planes(desc, cfg, q, xb, xs, dW, eng, ws_e,
                                                           None, st)
                fe()
                te = timed(fe, reps)
                ops = 2 * bits * macs
                row[tag] = {"ms": round(te, 5), "TOPS": round(ops / te / 1e9, 1),
                            "frac_of_peak": round(ops / te / 1e9 / peak, 4)}
                del ws_e
            print(json.dumps(row), flush=True)
            del X, dY, q, xwm, xb, xs, dW, dws
            torch.cuda.empty_cache()
        return

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
            # dY [K][M] ~ N(0,1) scaled per row by lognormal(0, 1.5)
            dY = _gen(torch, (K, M), torch.float32, dev,
                      torch.exp(1.5 * torch.randn((K, 1), device=dev)))
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
            # the quantizer at b = 4 with Bernoulli AGP on the same dY
            cfg4 = fqt.quant_cfg(4, fqt.FQT_AGP_BERNOULLI, 0, 0, 0)
            q4 = fqt.QGrad(desc, cfg4, device=dev)
            qws4 = fqt.workspace(desc, cfg4, fqt.FQT_WS_QUANTIZE, device=dev)
            qz4 = lambda: fqt.fqt_agp_scq_quantize(desc, cfg4, dY, q4, qws4, st)
            qz4()
            tq4 = timed(qz4, k)
            ops = 2.0 * M * M * K
            # quantize: dY read twice (statistics, codes) + 1-byte codes and b-bit planes of
            # both encodings written
            qbytes = K * M * 4 * 2 + 2 * K * M + 2 * K * M / 8
            print(json.dumps({"suite": name, "gemm_MxNxK": [M, M, K],
                              "gemm_dw_ms": round(tg, 4), "int8_TOPS": round(ops / tg / 1e9, 1),
                              "mfma_frac": round(ops / tg / 1e9 / MFMA_I8_PEAK_TOPS, 4),
                              "quantize_ms": round(tq, 4),
                              "quantize_GBps": round(qbytes / tq / 1e6, 1),
                              "quantize_b4_agp_ms": round(tq4, 4),
                              "quantize_b4_agp_GBps_of_dY_twice": round(K * M * 8 / tq4 / 1e6, 1),
                              "pack_x_ms": round(tp, 4)}), flush=True)
            del dY, X, q, qws, dws, xs, dW, q4, qws4
            torch.cuda.empty_cache()
        return

    out, _ = network_layers(name, dev, st, reps=reps, graph=True,
                            per_layer=lambda row: print(json.dumps(row), flush=True))
    print(json.dumps({"suite": name, "total_ms": out["ms_eager"],
                      "binary_TOPS": out["binary_TOPS_eager"], **out}), flush=True)


def calib_copy(torch, mib):
    """A plain device copy of `mib` MiB, three times, that counter runs scale by."""
    src = torch.ones(mib << 18, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    del src, dst


def main():
    args = parse()
    if args.suite:
        if args.gpus != 1:
            sys.exit("the suites run on one GPU")
        if args.calib_copy_mib:
            import torch
            calib_copy(torch, args.calib_copy_mib)
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
    stream = torch.cuda.current_stream()
    if args.calib_copy_mib:
        calib_copy(torch, args.calib_copy_mib)
    x, w, dy = draw_layer(layer, wl.recipe, wl.seed, wl.dtype)
    X, W, dY = (torch.from_numpy(a).to(dev) for a in (x, w, dy))
    dX, dW = torch.empty_like(X), torch.empty_like(W)
    desc = fqt.layer_desc(layer)
    cfg = fqt.quant_cfg(wl.bits, wl.agp_mode, wl.philox_seed, 0, 0)
    ws = fqt.workspace(desc, cfg, device=dev)
    macs = layer.binary_macs()
    ops_per_step = 2 * 2 * macs            # two products, 2 ops per binary MAC

    def step():
        fqt.fqt_layer_backward(desc, cfg, X, W, dY, dX, dW, ws, stream)

    for _ in range(args.warmup):
        step()
    ms_eager = _timed(torch, stream, step, args.steps)
    ms_graph = None
    # Graph mode: GRAPH_STEPS back-to-back steps per graph (as a network's step is one graph
    # of many layer calls), so that each replay's launch is shared by that many steps; the K
    # timed steps are K / GRAPH_STEPS replays (one step per graph when K is not a multiple).
    graph_steps = GRAPH_STEPS if args.steps % GRAPH_STEPS == 0 else 1
    if not args.no_graph:
        g = _graph_of(torch, stream,
                      lambda st: fqt.fqt_layer_backward(desc, cfg, X, W, dY, dX, dW, ws, st),
                      graph_steps)
        for _ in range(max(1, args.warmup // graph_steps)):
            g.replay()
        ms_graph = _timed(torch, stream, g.replay, args.steps // graph_steps) / graph_steps

    # Cold cache: before each timed step, overwrite 1 GiB (four times the last-level cache),
    # then time the step alone between two events.
    scrub = torch.empty(SCRUB_BYTES // 4, dtype=torch.float32, device=dev)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    cold_reps, cold_ms = max(5, min(50, args.steps // 4)), 0.0
    for r in range(cold_reps):
        scrub.fill_(float(r))
        e0.record(stream)
        step()
        e1.record(stream)
        torch.cuda.synchronize()
        cold_ms += e0.elapsed_time(e1)
    ms_cold = cold_ms / cold_reps
    del scrub

    warm = ms_eager if ms_graph is None else min(ms_eager, ms_graph)
    ms = ms_cold if args.cold else warm

    # The step's kernels through the entry points that launch them: the quantizer (statistics,
    # selection, codes), the two sign packers, and both products in one launch, the step's
    # longest kernel.  Each timed as a graph of REPS back-to-back launches replayed on
    # `stream` between two HIP events.
    q = fqt.QGrad(desc, cfg, device=dev)
    qws = fqt.workspace(desc, cfg, fqt.FQT_WS_QUANTIZE, device=dev)
    dws = fqt.workspace(desc, cfg, fqt.FQT_WS_GEMM_DW, device=dev)
    K = layer.C * layer.kh * layer.kw
    P = layer.Ho * layer.Wo
    R = layer.N * P
    HW = layer.H * layer.W
    Wd, Wr = (layer.D + 63) // 64, (R + 63) // 64
    xs = torch.empty(Wr * K, dtype=torch.int64, device=dev)
    wsb = torch.empty(K, 64 * Wd, dtype=torch.int8, device=dev)
    wls = torch.empty(K, dtype=torch.int32, device=dev)
    fqt.fqt_agp_scq_quantize(desc, cfg, dY, q, qws, stream)
    fqt.fqt_pack_input_signs(desc, X, xs, stream)
    fqt.fqt_pack_weight_signs(desc, W, wsb, wls, stream)
    entries = {
        "quantize": lambda st: fqt.fqt_agp_scq_quantize(desc, cfg, dY, q, qws, st),
        "pack_x": lambda st: fqt.fqt_pack_input_signs(desc, X, xs, st),
        "pack_w": lambda st: fqt.fqt_pack_weight_signs(desc, W, wsb, wls, st),
        "products": lambda st: fqt.fqt_binary_products(desc, cfg, q, xs, wsb, wls, dX, dW, dws,
                                                       st),
    }
    REPS = 20
    per = {}
    for name, fn in entries.items():
        if args.no_graph:
            for _ in range(args.warmup):
                fn(stream)
            per[name] = _timed(torch, stream, lambda: fn(stream), args.steps)
            continue
        gk = _graph_of(torch, stream, fn, REPS)
        for _ in range(max(1, args.warmup // REPS)):
            gk.replay()
        per[name] = _timed(torch, stream, gk.replay, max(1, args.steps // REPS)) / REPS
    torch.cuda.synchronize()
    ks, kc = int(q.psq_count.item()), int(q.pcq_count.item())
    b = wl.bits
    # Algorithmic bytes of the products launch: every operand crossing memory once at the
    # width the method needs (codes at b bits, signs at 1 bit) and the outputs.  Ops: the
    # int8 MFMA work over the kept rows (dX contracts D per kernel tap).
    code_bytes = (ks * P * layer.D + kc * R) * b / 8
    sign_bytes = (K * R + K * layer.D) / 8
    out_bytes = X.numel() * 4 + W.numel() * 4
    prod_bytes = code_bytes + sign_bytes + out_bytes
    prod_ops = 2 * ks * HW * K * layer.D + 2 * kc * K * R
    t_s = per["products"] * 1e-3
    if prod_bytes / (HBM_PEAK_GBS * 1e9) >= prod_ops / (MFMA_I8_PEAK_TOPS * 1e12):
        roofline = {"bound": "hbm", "achieved": prod_bytes / t_s / 1e9, "peak": HBM_PEAK_GBS,
                    "unit": "GB/s", "frac": prod_bytes / t_s / 1e9 / HBM_PEAK_GBS}
    else:
        roofline = {"bound": "mfma", "achieved": prod_ops / t_s / 1e12,
                    "peak": MFMA_I8_PEAK_TOPS, "unit": "TOPS",
                    "frac": prod_ops / t_s / 1e12 / MFMA_I8_PEAK_TOPS}
    roofline.update({"traffic": measured_traffic("products"), "kernel": "k_products",
                     "entry": "fqt_binary_products", "kernel_ms": per["products"],
                     "algorithmic_bytes": prod_bytes,
                     "algorithmic_bytes_parts": {"codes_b_bits": code_bytes,
                                                 "signs_1_bit": sign_bytes,
                                                 "dX_dW": out_bytes},
                     "int8_ops": prod_ops, "int8_frac": prod_ops / t_s / 1e12 / MFMA_I8_PEAK_TOPS,
                     "kept_samples": ks, "kept_channels": kc})
    # The whole step against HBM: dY, X, W read and dX, dW written once each.
    step_bytes = (dY.numel() + X.numel() + W.numel() + X.numel() + W.numel()) * 4
    step_roofline = {"bound": "hbm", "algorithmic_bytes": step_bytes,
                     "achieved": step_bytes / (ms * 1e-3) / 1e9, "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": step_bytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
                     "ms_at_peak": step_bytes / (HBM_PEAK_GBS * 1e9) * 1e3}

    # The single linear layer (32 x 256 -> 128, b = 2): launch-bound, eager and as a graph.
    wl1 = WORKLOADS["linear_32x256x128"]
    l1 = wl1.layers[0]
    x1, w1, dy1 = (torch.from_numpy(a).to(dev) for a in draw_layer(l1, wl1.recipe, wl1.seed))
    dx1, dw1 = torch.empty_like(x1), torch.empty_like(w1)
    d1 = fqt.layer_desc(l1)
    c1 = fqt.quant_cfg(wl1.bits, wl1.agp_mode, wl1.philox_seed, 0, 0)
    ws1 = fqt.workspace(d1, c1, device=dev)
    f1 = lambda st: fqt.fqt_layer_backward(d1, c1, x1, w1, dy1, dx1, dw1, ws1, st)
    for _ in range(args.warmup):
        f1(stream)
    cfg1 = {"workload": "linear_32x256x128", "ms_eager": _timed(torch, stream, lambda: f1(stream),
                                                                 args.steps)}
    if not args.no_graph:
        g1 = _graph_of(torch, stream, f1, 1)
        for _ in range(args.warmup):
            g1.replay()
        cfg1["ms_graph"] = _timed(torch, stream, g1.replay, args.steps)

    networks = None
    if not args.no_networks:
        networks = {n: network_layers(n, dev, stream, graph=not args.no_graph)[0]
                    for n in ("resnet18_32px", "vgg16_224_bf16")}

    cpu = None
    if not args.no_cpu_baseline:
        one, allc = cpu_legs(x, w, dy, layer, wl, ops_per_step, args.cpu_seconds)
        cpu = dict(one)
        cpu["all_cores"] = allc

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
                   "timed_as": "cold" if args.cold else (
                       "hip_graph" if ms_graph is not None and ms_graph <= ms_eager else "eager"),
                   "ms_per_step_eager": ms_eager, "ms_per_step_graph": ms_graph,
                   "graph_steps_per_replay": graph_steps,
                   "ms_per_step_cold": ms_cold, "per_entry_ms": per,
                   "binary_ops_per_step": ops_per_step,
                   "linear_32x256x128": cfg1, "networks": networks},
        "roofline": roofline,
        "step_roofline": step_roofline,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out))


if __name__ == "__main__":
    main()
