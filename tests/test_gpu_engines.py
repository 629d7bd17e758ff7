"""The dW product's popcount and fp4 engines (fqt_binary_gemm_dw_planes), which read the
PCQ bit planes and line-major sign bits, against the oracle: the integer I bit for bit,
dW within the rescale tolerance and bit-identical to the int8 engine's dW."""
import ctypes
import sys

import numpy as np
import pytest

from oracle import fqt as ofqt
from paper_2408_14267_amd.workloads import LayerShape, Recipe, draw_layer

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

CASES = [
    # name, layer, bits, AGP mode, recipe
    ("conv_ragged_b3", LayerShape("c", "conv2d", 5, 7, 70, 9, 9, 3, 3, 1, 1, 1, 1), 3, 0,
     Recipe("sample_lognormal", sigma=1.5)),
    ("conv_s2_b2", LayerShape("c", "conv2d", 6, 16, 32, 11, 11, 3, 3, 2, 2, 1, 1), 2, 0,
     Recipe("channel_lognormal", sigma=1.5)),
    ("vgg_cifar_conv_b4", LayerShape("conv", "conv2d", 128, 256, 256, 8, 8, 3, 3, 1, 1, 1, 1), 4,
     0, Recipe("sample_lognormal", sigma=2.0, outlier_count=13)),
    ("linear_b1_off", LayerShape("fc", "linear", 200, 300, 130), 1, 2,
     Recipe("sample_lognormal", sigma=1.0)),
    ("linear_ragged_b8", LayerShape("fc", "linear", 37, 300, 77), 8, 0,
     Recipe("sample_lognormal", sigma=2.0)),
    ("linear_b4_topk", LayerShape("fc", "linear", 64, 512, 128), 4, 1,
     Recipe("channel_lognormal", sigma=1.0)),
]


def _announce(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _inputs(fqt, layer, bits, mode, recipe, seed=0):
    x, w, dy = draw_layer(layer, recipe, seed)
    ref = ofqt.layer_backward(x, w, dy, bits, mode, seed=3, step=1, layer_id=2,
                              stride=layer.stride, pad=layer.pad)
    desc = fqt.layer_desc(layer)
    cfg = fqt.quant_cfg(bits, mode, 3, 1, 2)
    X, dY = torch.from_numpy(x).cuda(), torch.from_numpy(dy).cuda()
    q = fqt.QGrad(desc, cfg)
    fqt.fqt_agp_scq_quantize(desc, cfg, dY, q, fqt.workspace(desc, cfg, fqt.FQT_WS_QUANTIZE))
    K = layer.C * layer.kh * layer.kw
    Wr = (layer.N * layer.Ho * layer.Wo + 63) // 64
    xb = torch.empty(K * Wr, dtype=torch.int64, device="cuda")
    xs = torch.empty(K, dtype=torch.int32, device="cuda")
    if layer.kind == "linear":
        fqt.fqt_pack_bits(X, fqt.FQT_F32, layer.N, layer.C, layer.C, fqt.FQT_PACK_ALONG_ROWS, None,
                          xb, xs)
    else:
        fqt.fqt_pack_bits(X, fqt.FQT_F32, 0, 0, 0, fqt.FQT_PACK_IM2COL, desc, xb, xs)
    return ref, desc, cfg, X, q, xb, xs


@pytest.mark.parametrize("engine", ["popcount", "fp4"])
@pytest.mark.parametrize("name,layer,bits,mode,recipe", CASES, ids=[c[0] for c in CASES])
def test_engine_matches_oracle(engine, name, layer, bits, mode, recipe):
    from paper_2408_14267_amd import fqt
    if engine == "fp4" and bits > 4:
        pytest.skip("the fp4 engine takes b <= 4 (float32 sums of at most four planes)")
    _announce(f"[gpu engines] {engine} {name}: {layer} b={bits}")
    eng = fqt.FQT_ENGINE_POPCOUNT if engine == "popcount" else fqt.FQT_ENGINE_FP4
    ref, desc, cfg, X, q, xb, xs = _inputs(fqt, layer, bits, mode, recipe)
    D, K = layer.D, layer.C * layer.kh * layer.kw
    dW = torch.full((D, K), 7.0, device="cuda")
    I = torch.full((D, K), 7, dtype=torch.int32, device="cuda")
    ws = fqt.workspace(desc, cfg, fqt.FQT_WS_DW_POPCOUNT if engine == "popcount"
                       else fqt.FQT_WS_DW_FP4)
    fqt.fqt_binary_gemm_dw_planes(desc, cfg, q, xb, xs, dW, eng, ws, I)
    torch.cuda.synchronize()
    assert np.array_equal(I.cpu().numpy(), ref.I_dw), "I"
    g = dW.cpu().numpy().astype(np.float64)
    t1, t2 = ref.dW_t1.reshape(D, K), ref.dW_t2.reshape(D, K)
    assert (np.abs(g - ref.dW.reshape(D, K)) <= 1e-5 * (np.abs(t1) + np.abs(t2)) + 1e-30).all()
    # The int8 engine's dW from the same quantized gradient: the same bits.
    xwm = torch.empty(K * ((layer.N * layer.Ho * layer.Wo + 63) // 64), dtype=torch.int64,
                      device="cuda")
    fqt.fqt_pack_input_signs(desc, X, xwm)
    dW8 = torch.empty_like(dW)
    fqt.fqt_binary_gemm_dw(desc, cfg, q, xwm, dW8, fqt.workspace(desc, cfg, fqt.FQT_WS_GEMM_DW))
    torch.cuda.synchronize()
    assert torch.equal(dW8.view(torch.int32), dW.view(torch.int32))


@pytest.mark.parametrize("engine", ["popcount", "fp4"])
def test_engine_gemm_sweep_point_against_int8_engine(engine):
    """A large point of the GEMM sweep (M = N = 4096, 16384-deep contraction, b = 1, AGP off):
    the engine's integers equal the int8 engine's (pinned to the oracle on sampled outputs at
    16384 cubed) in full, and 64 sampled outputs equal the oracle's loop."""
    from oracle.philox import STREAM_ELEM, uniform_words
    from paper_2408_14267_amd import fqt
    M, Kc = 4096, 16384
    layer = LayerShape("g", "linear", Kc, M, M)
    _announce(f"[gpu engines] {engine} sweep point {M}x{M}x{Kc}")
    eng = fqt.FQT_ENGINE_POPCOUNT if engine == "popcount" else fqt.FQT_ENGINE_FP4
    gen = torch.Generator(device="cuda").manual_seed(4)
    dY = torch.randn((Kc, M), device="cuda", generator=gen)
    X = torch.randn((Kc, M), device="cuda", generator=gen)
    desc = fqt.layer_desc(layer)
    cfg = fqt.quant_cfg(1, fqt.FQT_AGP_OFF, 6, 0, 0)
    q = fqt.QGrad(desc, cfg)
    fqt.fqt_agp_scq_quantize(desc, cfg, dY, q, fqt.workspace(desc, cfg, fqt.FQT_WS_QUANTIZE))
    Wr = Kc // 64
    xb = torch.empty(M * Wr, dtype=torch.int64, device="cuda")
    xs = torch.empty(M, dtype=torch.int32, device="cuda")
    fqt.fqt_pack_bits(X, fqt.FQT_F32, Kc, M, M, fqt.FQT_PACK_ALONG_ROWS, None, xb, xs)
    xwm = torch.empty(M * Wr, dtype=torch.int64, device="cuda")
    fqt.fqt_pack_input_signs(desc, X, xwm)
    I8 = torch.empty((M, M), dtype=torch.int32, device="cuda")
    dW = torch.empty((M, M), device="cuda")
    fqt.fqt_binary_gemm_dw(desc, cfg, q, xwm, dW, fqt.workspace(desc, cfg, fqt.FQT_WS_GEMM_DW), I8)
    I = torch.empty_like(I8)
    ws = fqt.workspace(desc, cfg, fqt.FQT_WS_DW_POPCOUNT if engine == "popcount" else fqt.FQT_WS_DW_FP4)
    fqt.fqt_binary_gemm_dw_planes(desc, cfg, q, xb, xs, dW, eng, ws, I)
    torch.cuda.synchronize()
    assert torch.equal(I, I8)
    rng = np.random.default_rng(1)
    chans, cols = rng.choice(M, 8, replace=False), rng.choice(M, 8, replace=False)
    y = dY[:, torch.from_numpy(chans).cuda()].cpu().numpy()
    s = np.where(X[:, torch.from_numpy(cols).cuda()].cpu().numpy() > 0, 1, -1).astype(np.int64)
    n = np.arange(Kc, dtype=np.uint64)
    for a_, d in enumerate(chans):
        col = y[:, a_].astype(np.float32)
        u = uniform_words(n * np.uint64(M) + np.uint64(d), STREAM_ELEM, 6, 0, 0)
        qd = ofqt.sr_codes(col, col.min(), np.float32(col.max() - col.min()), 1, u).astype(np.int64)
        assert np.array_equal(I[int(d)][torch.from_numpy(cols).cuda()].cpu().numpy(), qd @ s)


def test_engine_rejections():
    from paper_2408_14267_amd import fqt
    layer = LayerShape("fc", "linear", 64, 64, 64)
    desc = fqt.layer_desc(layer)
    t = torch.empty(1 << 16, dtype=torch.int64, device="cuda")
    q = fqt.QGrad(desc, fqt.quant_cfg(8))
    p = ctypes.c_void_p(t.data_ptr())

    def call(d, cfg, eng):      # the C entry itself (the binding checks buffer sizes first)
        return fqt._lib.fqt_binary_gemm_dw_planes(ctypes.byref(d), ctypes.byref(cfg),
                                                  ctypes.byref(q.struct), p, p, p, None, eng, p,
                                                  t.numel() * 8, None)
    assert call(desc, fqt.quant_cfg(8), fqt.FQT_ENGINE_FP4) == fqt.FQT_E_INVAL
    assert call(desc, fqt.quant_cfg(2), 9) == fqt.FQT_E_INVAL
    big = fqt.layer_desc(LayerShape("fc", "linear", 16384, 8, 8))
    big.N, big.kind, big.H = 16384, fqt.FQT_CONV2D, 128         # 2^21 rows: 15 * 2^21 >= 2^24
    assert call(big, fqt.quant_cfg(4), fqt.FQT_ENGINE_FP4) == fqt.FQT_E_SHAPE
