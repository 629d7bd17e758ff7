"""GPU parity of the HIP path against the CPU oracle, through the C ABI.

Bit-exact: group selection (counts, kept-id partition), scale/offset/probability
bits, packed PSQ/PCQ planes, packed sign bits and line sums, and the integer
outputs of both products.  Rescaled float32 gradients: |gpu - oracle| <=
1e-5 * (|S I| + |Z' c|) elementwise (2^-8 for bfloat16 outputs), a bound that
stays meaningful where the two terms cancel.
"""
import sys
from dataclasses import replace

import numpy as np
import pytest

from oracle import fqt as ofqt
from paper_2408_14267_amd.workloads import WORKLOADS, LayerShape, Recipe, draw_layer

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def _fqt():
    from paper_2408_14267_amd import fqt
    return fqt


CASES = [
    # name, layer, bits, mode, recipe, dtype
    ("linear_32x256x128_b2", WORKLOADS["linear_32x256x128"].layers[0], 2, 0,
     WORKLOADS["linear_32x256x128"].recipe, "f32"),
    ("conv_ragged_b3", LayerShape("c", "conv2d", 5, 7, 70, 9, 9, 3, 3, 1, 1, 1, 1), 3, 0,
     Recipe("sample_lognormal", sigma=1.5), "f32"),
    ("conv_s2_b2", LayerShape("c", "conv2d", 6, 16, 32, 11, 11, 3, 3, 2, 2, 1, 1), 2, 0,
     Recipe("channel_lognormal", sigma=1.5), "f32"),
    ("conv1x1_s2_b4", LayerShape("c", "conv2d", 4, 64, 128, 8, 8, 1, 1, 2, 2, 0, 0), 4, 0,
     Recipe("student_t", df=3.0), "f32"),
    ("conv7x7_s2_b4", LayerShape("c", "conv2d", 4, 3, 64, 32, 32, 7, 7, 2, 2, 3, 3), 4, 0,
     Recipe("student_t", df=3.0), "f32"),
    # Sign forms of the selection launch on ragged shapes: a wave per 64 positions with a
    # partial channel group (3x3 and 1x1, stride 2, odd maps) and with W in another dtype.
    ("conv_s2_c6_oddmap_b3", LayerShape("c", "conv2d", 5, 6, 20, 9, 9, 3, 3, 2, 2, 1, 1), 3, 0,
     Recipe("channel_lognormal", sigma=1.0), "f32"),
    ("conv1x1_s2_c7_b2", LayerShape("c", "conv2d", 3, 7, 10, 7, 7, 1, 1, 2, 2, 0, 0), 2, 0,
     Recipe("sample_lognormal", sigma=1.0), "f32"),
    ("conv_s2_c10_bf16_b4", LayerShape("c", "conv2d", 4, 10, 24, 12, 12, 3, 3, 2, 2, 1, 1), 4,
     0, Recipe("student_t", df=3.0), "bf16"),
    ("linear_ragged_b8", LayerShape("fc", "linear", 37, 300, 77), 8, 0,
     Recipe("sample_lognormal", sigma=2.0), "f32"),
    ("linear_b1", LayerShape("fc", "linear", 64, 512, 128), 1, 0,
     Recipe("sample_lognormal", sigma=1.0), "f32"),
    ("conv_p49_b4", LayerShape("c", "conv2d", 3, 5, 8, 7, 7, 3, 3, 1, 1, 1, 1), 4, 0,
     Recipe("sample_lognormal", sigma=1.0), "f32"),
    ("conv_bf16_b2", LayerShape("c", "conv2d", 8, 32, 64, 14, 14, 3, 3, 1, 1, 1, 1), 2, 0,
     Recipe("channel_lognormal", sigma=1.5), "bf16"),
    ("conv_topk_b4", LayerShape("c", "conv2d", 16, 8, 24, 6, 6, 3, 3, 1, 1, 1, 1), 4, 1,
     Recipe("sample_lognormal", sigma=2.0), "f32"),
    ("conv_off_b2", LayerShape("c", "conv2d", 4, 8, 12, 5, 5, 3, 3, 1, 1, 1, 1), 2, 2,
     Recipe("sample_lognormal", sigma=1.0), "f32"),
    ("conv_1x1map_b4", LayerShape("c", "conv2d", 128, 16, 32, 1, 1, 3, 3, 1, 1, 1, 1), 4, 0,
     Recipe("student_t", df=3.0), "f32"),
    ("linear_N1_D1", LayerShape("fc", "linear", 1, 5, 1), 2, 0, Recipe(), "f32"),
    ("linear_wideD_b4", LayerShape("fc", "linear", 8, 64, 5000), 4, 0,
     Recipe("channel_lognormal", sigma=1.5), "f32"),
    ("conv5x5_b2", LayerShape("c", "conv2d", 3, 6, 40, 10, 10, 5, 5, 1, 1, 2, 2), 2, 0,
     Recipe("sample_lognormal", sigma=1.0), "f32"),
    ("conv2x3_mixed_stride_b3", LayerShape("c", "conv2d", 2, 5, 9, 6, 7, 2, 3, 1, 2, 0, 1), 3, 0,
     Recipe("channel_lognormal", sigma=1.0), "f32"),
    # 64 | Ho*Wo: the staged-band im2col path (ragged channel group, stride 2, bf16 input).
    ("conv_s2_p256_bf16_b4", LayerShape("c", "conv2d", 2, 20, 48, 32, 32, 3, 3, 2, 2, 1, 1), 4,
     0, Recipe("sample_lognormal", sigma=1.0), "bf16"),
    ("conv_p64_ragged_b2", LayerShape("c", "conv2d", 3, 33, 40, 8, 8, 3, 3, 1, 1, 1, 1), 2, 0,
     Recipe("channel_lognormal", sigma=1.0), "f32"),
    # Stride-1 same-padded kernels that are not square (bit-level im2col: 1x1, 1x3).
    ("conv1x1_s1_b2", LayerShape("c", "conv2d", 3, 20, 12, 5, 6, 1, 1, 1, 1, 0, 0), 2, 0,
     Recipe("sample_lognormal", sigma=1.0), "f32"),
    ("conv1x3_b3", LayerShape("c", "conv2d", 2, 5, 9, 6, 7, 1, 3, 1, 1, 0, 1), 3, 0,
     Recipe("channel_lognormal", sigma=1.0), "bf16"),
    # Sample ranges decaying geometrically: AGP saturation takes 8 rounds (the most the
    # selection runs) and 9 rounds (the selection falls back to sorting the weights).
    ("conv_geometric_8_rounds_b2", LayerShape("c", "conv2d", 96, 8, 40, 6, 6, 3, 3, 1, 1, 1, 1),
     2, 0, Recipe("sample_geometric", ratio=0.8), "f32"),
    ("conv_geometric_sorted_b3", LayerShape("c", "conv2d", 200, 8, 24, 6, 6, 3, 3, 1, 1, 1, 1),
     3, 0, Recipe("sample_geometric", ratio=0.8), "f32"),
    # 8x8 maps, odd batch, 256 channels: the sign packs in the selection launch.
    ("conv_p64_odd_batch_b4", LayerShape("c", "conv2d", 129, 256, 32, 8, 8, 3, 3, 1, 1, 1, 1),
     4, 0, Recipe("sample_lognormal", sigma=1.0), "f32"),
    # 65536 output pixels per sample: group partials reduced by a workgroup per group before
    # the selection; many dW splits with the block-per-row finish.
    ("conv_bigmap_b2", LayerShape("c", "conv2d", 2, 4, 16, 256, 256, 3, 3, 1, 1, 1, 1), 2, 0,
     Recipe("sample_lognormal", sigma=1.0), "f32"),
    ("conv_bigmap_8_samples_b2", LayerShape("c", "conv2d", 8, 4, 70, 256, 256, 3, 3, 1, 1, 1, 1),
     2, 0, Recipe("sample_lognormal", sigma=1.0), "f32"),
    # 524288 rows, b = 8: the long split-R dW partials, biased codes; about 5 kept channels
    # expected, so one row tile per wave.
    ("conv_bigmap_b8", LayerShape("c", "conv2d", 8, 4, 40, 256, 256, 3, 3, 1, 1, 1, 1), 8, 0,
     Recipe("channel_lognormal", sigma=1.0), "f32"),
    # The same long split-R partials with about 40 kept channels: two row tiles per wave.
    ("conv_bigmap_rt2_b2", LayerShape("c", "conv2d", 8, 4, 80, 256, 256, 3, 3, 1, 1, 1, 1), 2,
     0, Recipe("channel_lognormal", sigma=1.0), "f32"),
    # 16384 dX tiles of 32 x 32: the dX product in its four-tiles-per-block form.
    ("conv_wide_dx_b2", LayerShape("c", "conv2d", 4, 64, 8, 256, 256, 3, 3, 1, 1, 1, 1), 2, 0,
     Recipe("channel_lognormal", sigma=1.0), "f32"),
    # The same form on odd 297 x 297 maps with 40 channels: pixel tiles that straddle two
    # samples, rows that are not 16-byte aligned and the partial second channel tile take
    # the element-by-element stores, the rest the 16-byte ones.
    ("conv_wide_dx_oddmap_b2", LayerShape("c", "conv2d", 3, 40, 8, 297, 297, 3, 3, 1, 1, 1, 1),
     2, 0, Recipe("channel_lognormal", sigma=1.0), "f32"),
    # Large one-split dW outputs: the 2 x 2-tile dW form (ragged sizes, b = 8 bias).
    ("linear_bigdw_b2", LayerShape("fc", "linear", 64, 2048, 2048), 2, 0,
     Recipe("channel_lognormal", sigma=1.5), "f32"),
    ("linear_bigdw_ragged_b8", LayerShape("fc", "linear", 100, 2100, 2050), 8, 0,
     Recipe("sample_lognormal", sigma=1.0), "f32"),
    # AGP off with more than 1024 samples: the per-group selection over the whole chip;
    # channel-fast statistics and codes; one-bit codes; the big dW form with AGP off.
    ("linear_off_large_b1", LayerShape("fc", "linear", 2048, 96, 1300), 1, 2,
     Recipe("sample_lognormal", sigma=1.0), "f32"),
    ("linear_bigdw_off_b1", LayerShape("fc", "linear", 256, 2048, 2112), 1, 2,
     Recipe("channel_lognormal", sigma=1.0), "f32"),
    # Big dW forms over contractions of 8 words and more (the long form's word ring, with
    # a ragged last word and the b = 8 bias).
    ("linear_bigdw_long_b2", LayerShape("fc", "linear", 520, 2048, 2048), 2, 0,
     Recipe("channel_lognormal", sigma=1.5), "f32"),
    ("linear_bigdw_long_ragged_b8", LayerShape("fc", "linear", 600, 2100, 2050), 8, 0,
     Recipe("sample_lognormal", sigma=1.0), "f32"),
    # More than 1024 samples with geometrically decaying ranges: the many-group selection
    # saturates in 6 rounds, and (9 rounds needed) falls back to its sort.
    ("linear_geometric_large_6_rounds_b2", LayerShape("fc", "linear", 1500, 8, 40), 2, 0,
     Recipe("sample_geometric", ratio=0.99), "f32"),
    ("linear_geometric_large_sorted_b3", LayerShape("fc", "linear", 1500, 8, 40), 3, 0,
     Recipe("sample_geometric", ratio=0.97), "f32"),
]


# The layers of the benchmarked networks at their real shapes.
_CH15 = Recipe("channel_lognormal", sigma=1.5)
_VGG = {L.name: L for L in WORKLOADS["vgg16_224_bf16"].layers}
WORKLOAD_CASES = [
    # VGG-16 at 224 x 224 (bf16 x / dy / dx, b = 2, per-channel lognormal(0, 1.5) scale), at
    # batch 2: maps of 224^2 and 112^2 pixels take the per-plane statistics in bf16.
    ("vgg16_224_conv1_n2_bf16", replace(_VGG["conv1"], N=2),
     2, 0, _CH15, "bf16"),
    ("vgg16_224_conv2_n2_bf16", replace(_VGG["conv2"], N=2),
     2, 0, _CH15, "bf16"),
    ("vgg16_224_conv3_n2_bf16", replace(_VGG["conv3"], N=2),
     2, 0, _CH15, "bf16"),
    # 16384 dX tiles with bf16 output: the dX product's four-tiles-per-block form in bf16.
    ("conv_wide_dx_bf16_b2", LayerShape("c", "conv2d", 4, 64, 8, 256, 256, 3, 3, 1, 1, 1, 1), 2,
     0, _CH15, "bf16"),
    ("conv_wide_dx_oddmap_bf16_b4", LayerShape("c", "conv2d", 3, 64, 8, 297, 297, 3, 3, 1, 1, 1,
                                                1), 4, 0, _CH15, "bf16"),
    # A point of the binary GEMM sweep as a layer (M = N = 1024, K = 2304 rows) at b = 4 with
    # Bernoulli AGP.
    ("gemm_sweep_1024x1024x2304_b4", LayerShape("g", "linear", 2304, 1024, 1024), 4, 0,
     Recipe("sample_lognormal", sigma=1.5), "f32"),
]
# Every layer of ResNet-18 (ImageNet stem) at 32 x 32, batch 128, b = 4, Student-t(3) dY drawn
# with data seed = layer index, as the network suite runs it.
RESNET_CASES = [(f"resnet18_{i:02d}_{L.name}", L, i) for i, L in
                enumerate(WORKLOADS["resnet18_32px"].layers)]


def _announce(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _to_dev(a, dtype):
    t = torch.from_numpy(np.ascontiguousarray(a)).cuda()
    return t.to(torch.bfloat16) if dtype == "bf16" else t


def _u64(t):
    return t.cpu().numpy().view(np.uint64)


def _bits32(a):
    return np.asarray(a, dtype=np.float32).view(np.uint32)


def _assert_rescaled(got, ref, t1, t2, rel, what):
    g = got.float().cpu().numpy().astype(np.float64).reshape(ref.shape)
    bound = rel * (np.abs(t1) + np.abs(t2)) + 1e-30
    bad = np.abs(g - ref) > bound
    assert not bad.any(), f"{what}: {int(bad.sum())} of {bad.size} outside tolerance; " \
                          f"first at {np.argwhere(bad)[0]}"


def _run_case(layer, bits, mode, recipe, dtype, seed=0, step=3, layer_id=5, data_seed=0):
    fqt = _fqt()
    x, w, dy = draw_layer(layer, recipe, data_seed, dtype)
    ref = ofqt.layer_backward(x, w, dy, bits, mode, seed=seed, step=step, layer_id=layer_id,
                              stride=layer.stride, pad=layer.pad)
    dt = fqt.FQT_BF16 if dtype == "bf16" else fqt.FQT_F32
    desc = fqt.layer_desc(layer, dy_dtype=dt, x_dtype=dt, w_dtype=fqt.FQT_F32, dx_dtype=dt)
    cfg = fqt.quant_cfg(bits, mode, seed, step, layer_id)
    X, W, dY = _to_dev(x, dtype), _to_dev(w, "f32"), _to_dev(dy, dtype)
    return fqt, ref, desc, cfg, X, W, dY


def _rows_of_chunks(t, rows, chunks):
    """[chunks][rows][32] bytes on the device -> [rows][32 * chunks] on the host."""
    return t.cpu().numpy().reshape(chunks, rows, 32).transpose(1, 0, 2).reshape(rows, 32 * chunks)


def _check_quantize(fqt, ref, desc, cfg, dY, layer, bits):
    q = fqt.QGrad(desc, cfg)
    ws = fqt.workspace(desc, cfg, fqt.FQT_WS_QUANTIZE)
    fqt.fqt_agp_scq_quantize(desc, cfg, dY, q, ws)
    torch.cuda.synchronize()
    N, D, P = layer.N, layer.D, layer.Ho * layer.Wo
    R = N * P
    Wd, Wr = (D + 63) // 64, (R + 63) // 64
    for name, grp, kept, count, scale, offset, prob in (
            ("samples", ref.qgrad.samples, q.psq_kept, q.psq_count, q.psq_scale, q.psq_offset,
             q.psq_prob),
            ("channels", ref.qgrad.channels, q.pcq_kept, q.pcq_count, q.pcq_scale, q.pcq_offset,
             q.pcq_prob)):
        assert int(count.item()) == grp.count, name
        assert np.array_equal(kept.cpu().numpy(), grp.kept_ids), name
        assert np.array_equal(_bits32(prob.cpu().numpy()), _bits32(grp.prob)), name + " prob"
        assert np.array_equal(_bits32(scale.cpu().numpy()), _bits32(grp.scale)), name + " scale"
        assert np.array_equal(_bits32(offset.cpu().numpy()), _bits32(grp.offset)), name + " offset"
    ks, kc = ref.qgrad.samples.count, ref.qgrad.channels.count
    psq = _u64(q.psq_planes).reshape(bits, R, Wd)[:, :ks * P]
    pcq = _u64(q.pcq_planes).reshape(bits, D, Wr)[:, :kc]
    assert np.array_equal(psq, ref.qgrad.psq_planes), "psq planes"
    assert np.array_equal(pcq, ref.qgrad.pcq_planes), "pcq planes"
    # Code arrays are chunk-major ([32-byte chunk][row][32]); back to rows for the check.
    psq_codes = _rows_of_chunks(q.psq_codes, R, 2 * Wd)[:ks * P]
    pcq_codes = _rows_of_chunks(q.pcq_codes, D, 2 * Wr)[:kc]
    assert np.array_equal(psq_codes[:, :D], ref.qgrad.psq_rows), "psq codes"
    assert not psq_codes[:, D:].any(), "psq code padding"
    assert np.array_equal(pcq_codes[:, :R], ref.qgrad.pcq_rows), "pcq codes"
    assert not pcq_codes[:, R:].any(), "pcq code padding"
    return q


def _check_signs(fqt, ref, desc, layer, X, W, x_dt):
    K = layer.C * layer.kh * layer.kw
    R = layer.N * layer.Ho * layer.Wo
    Wd, Wr = (layer.D + 63) // 64, (R + 63) // 64
    xs = torch.empty(K * Wr, dtype=torch.int64, device="cuda")
    xsum = torch.empty(K, dtype=torch.int32, device="cuda")
    ws_ = torch.empty(K * Wd, dtype=torch.int64, device="cuda")
    wsum = torch.empty(K, dtype=torch.int32, device="cuda")
    if layer.kind == "linear":
        fqt.fqt_pack_bits(X, x_dt, layer.N, layer.C, layer.C, fqt.FQT_PACK_ALONG_ROWS, None, xs, xsum)
    else:
        fqt.fqt_pack_bits(X, x_dt, 0, 0, 0, fqt.FQT_PACK_IM2COL, desc, xs, xsum)
    fqt.fqt_pack_bits(W, fqt.FQT_F32, layer.D, K, K, fqt.FQT_PACK_ALONG_ROWS, None, ws_, wsum)
    wsb = torch.empty(K, 64 * Wd, dtype=torch.int8, device="cuda")
    wlsum = torch.empty(K, dtype=torch.int32, device="cuda")
    fqt.fqt_pack_weight_signs(desc, W, wsb, wlsum)
    xwm = torch.empty(Wr, K, dtype=torch.int64, device="cuda")
    fqt.fqt_pack_input_signs(desc, X, xwm)
    torch.cuda.synchronize()
    # The dW operand: the same im2col bits, word-major.
    assert np.array_equal(_u64(xwm), ofqt.pack_words(ref.xbits).T), "x sign words (word-major)"
    assert np.array_equal(_u64(xs).reshape(K, Wr), ofqt.pack_words(ref.xbits)), "x sign bits"
    assert np.array_equal(_u64(ws_).reshape(K, Wd), ofqt.pack_words(ref.wbits)), "w sign bits"
    assert np.array_equal(xsum.cpu().numpy(), ref.xsign_colsum), "x line sums"
    assert np.array_equal(wsum.cpu().numpy(), ref.wsign_colsum), "w line sums"
    # The +-1 byte form of sign(W): the oracle's sign bits as +1 / -1, zero past D, stored
    # [32-byte chunk of D][tap][channel][32].
    taps = layer.kh * layer.kw
    want = np.zeros((K, 64 * Wd), dtype=np.int8)
    want[:, :layer.D] = np.where(ref.wbits, 1, -1)
    want = want.reshape(layer.C, taps, 2 * Wd, 32).transpose(2, 1, 0, 3)
    assert np.array_equal(wsb.cpu().numpy().reshape(2 * Wd, taps, layer.C, 32), want), \
        "w sign bytes"
    assert np.array_equal(wlsum.cpu().numpy(), ref.wsign_colsum), "w sign-byte line sums"
    return xwm, xsum, wsb, wlsum


@pytest.mark.parametrize("name,layer,bits,mode,recipe,dtype", CASES, ids=[c[0] for c in CASES])
def test_kernels_match_oracle(name, layer, bits, mode, recipe, dtype):
    _announce(f"[gpu parity] {name}: {layer} b={bits} mode={mode} {dtype}")
    _check_case(layer, bits, mode, recipe, dtype)


def _check_case(layer, bits, mode, recipe, dtype, **kw):
    fqt, ref, desc, cfg, X, W, dY = _run_case(layer, bits, mode, recipe, dtype, **kw)
    x_dt = fqt.FQT_BF16 if dtype == "bf16" else fqt.FQT_F32
    q = _check_quantize(fqt, ref, desc, cfg, dY, layer, bits)
    xs, xsum, wsb, wlsum = _check_signs(fqt, ref, desc, layer, X, W, x_dt)
    D, K = layer.D, layer.C * layer.kh * layer.kw
    dW = torch.empty(D, K, dtype=torch.float32, device="cuda")
    I_dw = torch.empty(D, K, dtype=torch.int32, device="cuda")
    fqt.fqt_binary_gemm_dw(desc, cfg, q, xs, dW, fqt.workspace(desc, cfg, fqt.FQT_WS_GEMM_DW), I_dw)
    dX = torch.empty(X.shape, dtype=X.dtype, device="cuda")
    I_dx = torch.empty(layer.N, layer.C, layer.H, layer.W, dtype=torch.int32, device="cuda")
    fqt.fqt_binary_gemm_dx(desc, cfg, q, wsb, wlsum, dX, I_dx)
    torch.cuda.synchronize()
    assert np.array_equal(I_dw.cpu().numpy(), ref.I_dw), "dW integer product"
    assert np.array_equal(I_dx.cpu().numpy(), ref.I_dx), "dX integer product"
    _assert_rescaled(dW, ref.dW, ref.dW_t1, ref.dW_t2, 1e-5, "dW")
    _assert_rescaled(dX, ref.dX, ref.dX_t1, ref.dX_t2, 2.0 ** -8 if dtype == "bf16" else 1e-5, "dX")
    # Both products in one launch (fqt_binary_products) give the same bits as the two calls.
    dX3, dW3 = torch.full_like(dX, 7.0), torch.full_like(dW, 7.0)
    fqt.fqt_binary_products(desc, cfg, q, xs, wsb, wlsum, dX3, dW3,
                            fqt.workspace(desc, cfg, fqt.FQT_WS_GEMM_DW))
    torch.cuda.synchronize()
    assert torch.equal(dX3.view(torch.int16 if dtype == "bf16" else torch.int32),
                       dX.view(torch.int16 if dtype == "bf16" else torch.int32)), "products dX"
    assert torch.equal(dW3.view(torch.int32), dW.view(torch.int32)), "products dW"
    # The whole-layer entry point (the launch configuration of the network suites) gives the
    # same bits as the component calls.
    dX2 = torch.empty_like(dX)
    dW2 = torch.empty_like(dW)
    fqt.fqt_layer_backward(desc, cfg, X, W, dY, dX2, dW2, fqt.workspace(desc, cfg))
    torch.cuda.synchronize()
    assert torch.equal(dX2.view(torch.int16 if dtype == "bf16" else torch.int32),
                       dX.view(torch.int16 if dtype == "bf16" else torch.int32))
    assert torch.equal(dW2.view(torch.int32), dW.view(torch.int32))
    return ref


@pytest.mark.parametrize("name,layer,bits,mode,recipe,dtype", WORKLOAD_CASES,
                         ids=[c[0] for c in WORKLOAD_CASES])
def test_workload_layers_match_oracle(name, layer, bits, mode, recipe, dtype):
    """Layers of the benchmarked configurations at their real geometry (smaller batch where
    the oracle needs it), compared element by element as in test_kernels_match_oracle."""
    _announce(f"[gpu parity] workload layer {name}: {layer} b={bits} {dtype}")
    _check_case(layer, bits, mode, recipe, dtype)


@pytest.mark.parametrize("name,layer,index", RESNET_CASES, ids=[c[0] for c in RESNET_CASES])
def test_resnet18_layers_match_oracle(name, layer, index):
    """Every ResNet-18 layer at batch 128 (the network suite's shapes, dY drawn as it draws
    them: Student-t(3), data seed and layer id = layer index), compared in full."""
    wl = WORKLOADS["resnet18_32px"]
    _announce(f"[gpu parity] {name}: {layer}")
    _check_case(layer, wl.bits, wl.agp_mode, wl.recipe, wl.dtype, seed=wl.philox_seed, step=0,
                layer_id=index, data_seed=index)


def test_vgg16_fc6_bf16_sampled():
    """VGG-16 fc6 (25088 -> 4096, batch 64, bf16 x / dy / dx, b = 2, per-channel lognormal
    dY) through fqt_layer_backward: the selection, scales and codes bit for bit, dX in full,
    and dW on 16 sampled output channels (kept and pruned, first and last), against the
    oracle's rows for those channels."""
    fqt = _fqt()
    wl = WORKLOADS["vgg16_224_bf16"]
    layer = _VGG["fc6"]
    _announce(f"[gpu parity] fc6 sampled: {layer}")
    x, w, dy = draw_layer(layer, wl.recipe, 6, "bf16")
    bits, seed, step, lid = wl.bits, 3, 1, 13
    qref = ofqt.agp_scq_quantize(dy, bits, wl.agp_mode, seed, step, lid)
    ch = qref.channels
    kept, pruned = ch.kept_ids[:ch.count], ch.kept_ids[ch.count:]
    assert kept.size >= 7 and pruned.size >= 7
    chans = np.unique(np.concatenate([[0, layer.D - 1], kept[:7], pruned[:7]]))
    ref = ofqt.layer_backward(x, w, dy, bits, wl.agp_mode, seed=seed, step=step, layer_id=lid,
                              dw_channels=chans)
    desc = fqt.layer_desc(layer, fqt.FQT_BF16, fqt.FQT_BF16, fqt.FQT_F32, fqt.FQT_BF16)
    cfg = fqt.quant_cfg(bits, wl.agp_mode, seed, step, lid)
    X, W, dY = _to_dev(x, "bf16"), _to_dev(w, "f32"), _to_dev(dy, "bf16")
    _check_quantize(fqt, ref, desc, cfg, dY, layer, bits)
    dX = torch.empty(X.shape, dtype=torch.bfloat16, device="cuda")
    dW = torch.empty(W.shape, dtype=torch.float32, device="cuda")
    fqt.fqt_layer_backward(desc, cfg, X, W, dY, dX, dW, fqt.workspace(desc, cfg))
    torch.cuda.synchronize()
    _assert_rescaled(dX, ref.dX, ref.dX_t1, ref.dX_t2, 2.0 ** -8, "dX")
    rows = dW[torch.from_numpy(chans).cuda()]
    _assert_rescaled(rows, ref.dW, ref.dW_t1, ref.dW_t2, 1e-5, "dW sampled rows")
    assert not rows[torch.from_numpy(~np.isin(chans, kept)).cuda()].any(), "pruned dW rows"


def test_full_vgg_cifar_conv_layer():
    """The benchmarked workload (VGG-16 CIFAR 3x3 conv 256->256 on 8x8, N=128, b=4) in the
    launch configuration the benchmark times, compared in full."""
    wl = WORKLOADS["vgg_cifar_conv3x3_256"]
    layer = wl.layers[0]
    _announce(f"[gpu parity] full {wl.name}")
    fqt, ref, desc, cfg, X, W, dY = _run_case(layer, wl.bits, wl.agp_mode, wl.recipe, wl.dtype,
                                             seed=wl.philox_seed, step=0, layer_id=0,
                                             data_seed=wl.seed)
    _check_quantize(fqt, ref, desc, cfg, dY, layer, wl.bits)
    dX = torch.empty_like(X)
    dW = torch.empty_like(W)
    ws = fqt.workspace(desc, cfg)
    for _ in range(2):      # a repeated call on a reused workspace gives the same result
        fqt.fqt_layer_backward(desc, cfg, X, W, dY, dX, dW, ws)
        torch.cuda.synchronize()
        _assert_rescaled(dW, ref.dW, ref.dW_t1, ref.dW_t2, 1e-5, "dW")
        _assert_rescaled(dX, ref.dX, ref.dX_t1, ref.dX_t2, 1e-5, "dX")
    assert 0 < ref.qgrad.samples.count < layer.N and 0 < ref.qgrad.channels.count < layer.D


def test_dw_product_16384_cube_sampled():
    """The dW product at 16384 x 16384 over a 16384-deep contraction (the large GEMM sweep's
    largest point: the long big-dW form, a 256-word contraction), b = 1, AGP off, on sampled
    outputs: the integer I of 8 channels x 64 columns from the oracle's own quantizer steps on
    those channels (statistics, Philox words, stochastic rounding) and the sign bits of those
    columns of X; dW within the rescale tolerance."""
    from oracle.philox import STREAM_ELEM, uniform_words
    fqt = _fqt()
    N = C = D = 16384
    seed, step, lid = 7, 1, 2
    layer = LayerShape("fc", "linear", N, C, D)
    _announce(f"[gpu parity] sampled dW {layer}")
    gen = torch.Generator(device="cuda").manual_seed(11)
    dY = torch.randn((N, D), device="cuda", generator=gen)
    X = torch.randn((N, C), device="cuda", generator=gen)
    desc = fqt.layer_desc(layer)
    cfg = fqt.quant_cfg(1, fqt.FQT_AGP_OFF, seed, step, lid)
    q = fqt.QGrad(desc, cfg)
    fqt.fqt_agp_scq_quantize(desc, cfg, dY, q, fqt.workspace(desc, cfg, fqt.FQT_WS_QUANTIZE))
    xs = torch.empty(((N + 63) // 64) * C, dtype=torch.int64, device="cuda")
    fqt.fqt_pack_input_signs(desc, X, xs)
    dW = torch.empty((D, C), dtype=torch.float32, device="cuda")
    I_dw = torch.empty((D, C), dtype=torch.int32, device="cuda")
    fqt.fqt_binary_gemm_dw(desc, cfg, q, xs, dW, fqt.workspace(desc, cfg, fqt.FQT_WS_GEMM_DW), I_dw)
    torch.cuda.synchronize()
    rng = np.random.default_rng(5)
    chans = np.concatenate([[0, D - 1], rng.choice(D, 6, replace=False)])
    cols = np.concatenate([[0, C - 1], rng.choice(C, 62, replace=False)])
    y = dY[:, torch.from_numpy(chans).cuda()].cpu().numpy()           # [N][8]
    xb = (X[:, torch.from_numpy(cols).cuda()].cpu().numpy() > 0)       # [N][64]
    s = np.where(xb, 1, -1).astype(np.int64)
    I_got = I_dw[torch.from_numpy(chans).cuda()][:, torch.from_numpy(cols).cuda()].cpu().numpy()
    W_got = dW[torch.from_numpy(chans).cuda()][:, torch.from_numpy(cols).cuda()].cpu().numpy()
    n = np.arange(N, dtype=np.uint64)
    for a, d in enumerate(chans):
        col = y[:, a].astype(np.float32)
        Z = col.min()
        R = np.float32(col.max() - Z)
        u32 = uniform_words(n * np.uint64(D) + np.uint64(d), STREAM_ELEM, seed, step, lid)
        qd = ofqt.sr_codes(col, Z, R, 1, u32).astype(np.int64)
        I_ref = qd @ s                                                 # [64]
        assert np.array_equal(I_got[a], I_ref), f"I of channel {d}"
        # AGP off: S = R / B, Z' = Z; c = 2 T - N over the column's set bits.
        S = np.float32(np.float64(R) / 1.0)
        c = (2 * xb.sum(axis=0) - N).astype(np.float64)
        t1, t2 = np.float64(S) * I_ref, np.float64(Z) * c
        bad = np.abs(W_got[a].astype(np.float64) - (t1 + t2)) > 1e-5 * (np.abs(t1) + np.abs(t2)) + 1e-30
        assert not bad.any(), f"dW of channel {d}"


def test_layer_backward_graph_replays_match_eager():
    """fqt_layer_backward captured in a HIP graph on a side stream and replayed several
    times, with eager calls on other data and synchronizations between the replays: every
    replay equals the eager result bit for bit."""
    wl = WORKLOADS["resnet18_32px"]
    layer = wl.layers[3]
    _announce(f"[gpu parity] graph replay {layer}")
    fqt = _fqt()
    desc = fqt.layer_desc(layer)
    cfg = fqt.quant_cfg(wl.bits, wl.agp_mode, 11, 2, 1)
    X, W, dY = (_to_dev(a, "f32") for a in draw_layer(layer, wl.recipe, 1, "f32"))
    X2, W2, dY2 = (_to_dev(a, "f32") for a in draw_layer(layer, wl.recipe, 2, "f32"))
    ws, ws2 = fqt.workspace(desc, cfg), fqt.workspace(desc, cfg)
    dX_e, dW_e = torch.empty_like(X), torch.empty_like(W)
    fqt.fqt_layer_backward(desc, cfg, X, W, dY, dX_e, dW_e, ws)
    torch.cuda.synchronize()
    dX_g, dW_g = torch.empty_like(X), torch.empty_like(W)
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        with torch.cuda.graph(g, stream=side):
            fqt.fqt_layer_backward(desc, cfg, X, W, dY, dX_g, dW_g, ws, side)
    torch.cuda.synchronize()
    dX_o, dW_o = torch.empty_like(X2), torch.empty_like(W2)
    for r in range(3):
        dX_g.fill_(7.0)
        dW_g.fill_(7.0)
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(dX_g.view(torch.int32), dX_e.view(torch.int32)), f"replay {r} dX"
        assert torch.equal(dW_g.view(torch.int32), dW_e.view(torch.int32)), f"replay {r} dW"
        fqt.fqt_layer_backward(desc, cfg, X2, W2, dY2, dX_o, dW_o, ws2)   # eager work between
        torch.cuda.synchronize()


def test_all_zero_gradient():
    fqt = _fqt()
    layer = LayerShape("c", "conv2d", 4, 8, 16, 6, 6, 3, 3, 1, 1, 1, 1)
    _announce("[gpu parity] all-zero dY")
    x, w, _ = draw_layer(layer, Recipe(), 0)
    desc = fqt.layer_desc(layer)
    cfg = fqt.quant_cfg(4)
    X, W = _to_dev(x, "f32"), _to_dev(w, "f32")
    dY = torch.zeros(layer.dy_shape, device="cuda")
    dX = torch.full_like(X, 7.0)
    dW = torch.full_like(W, 7.0)
    fqt.fqt_layer_backward(desc, cfg, X, W, dY, dX, dW, fqt.workspace(desc, cfg))
    torch.cuda.synchronize()
    assert torch.count_nonzero(dX).item() == 0 and torch.count_nonzero(dW).item() == 0


def test_constant_gradient_exact_with_agp_off():
    fqt = _fqt()
    layer = LayerShape("fc", "linear", 16, 40, 24)
    _announce("[gpu parity] constant dY, AGP off")
    x, w, _ = draw_layer(layer, Recipe(), 0)
    dy = np.full(layer.dy_shape, 0.75, np.float32)
    desc = fqt.layer_desc(layer)
    cfg = fqt.quant_cfg(2, fqt.FQT_AGP_OFF)
    X, W, dY = (_to_dev(a, "f32") for a in (x, w, dy))
    dX, dW = torch.empty_like(X), torch.empty_like(W)
    fqt.fqt_layer_backward(desc, cfg, X, W, dY, dX, dW, fqt.workspace(desc, cfg))
    torch.cuda.synchronize()
    sx, sw = np.where(x > 0, 1.0, -1.0), np.where(w > 0, 1.0, -1.0)
    np.testing.assert_allclose(dW.cpu().numpy(), dy.T.astype(np.float64) @ sx, rtol=1e-6)
    np.testing.assert_allclose(dX.cpu().numpy(), dy.astype(np.float64) @ sw, rtol=1e-6)


def test_seed_step_layer_change_the_draws():
    fqt = _fqt()
    layer = LayerShape("fc", "linear", 32, 64, 48)
    _announce("[gpu parity] seeds")
    x, w, dy = draw_layer(layer, Recipe("sample_lognormal", sigma=1.0), 0)
    desc = fqt.layer_desc(layer)
    outs = []
    for seed, step, lid in ((0, 0, 0), (1, 0, 0), (0, 1, 0), (0, 0, 1)):
        cfg = fqt.quant_cfg(2, 0, seed, step, lid)
        X, W, dY = (_to_dev(a, "f32") for a in (x, w, dy))
        dX, dW = torch.empty_like(X), torch.empty_like(W)
        fqt.fqt_layer_backward(desc, cfg, X, W, dY, dX, dW, fqt.workspace(desc, cfg))
        torch.cuda.synchronize()
        ref = ofqt.layer_backward(x, w, dy, 2, 0, seed=seed, step=step, layer_id=lid)
        _assert_rescaled(dX, ref.dX, ref.dX_t1, ref.dX_t2, 1e-5, "dX")
        outs.append(dX.cpu())
    assert all(not torch.equal(outs[0], o) for o in outs[1:])


def test_workspace_shared_across_layers():
    """One zero-filled workspace, sized for the largest of several layers, serves them in
    turn (twice over): every call matches the oracle and leaves the workspace's state bytes
    (the merged group keys) zero."""
    fqt = _fqt()
    layers = [
        (LayerShape("c", "conv2d", 5, 7, 70, 9, 9, 3, 3, 1, 1, 1, 1), 3,
         Recipe("sample_lognormal", sigma=1.5)),
        (LayerShape("fc", "linear", 37, 300, 77), 8, Recipe("sample_lognormal", sigma=2.0)),
        # 32 x 32 maps: per-plane statistics, no merged keys
        (LayerShape("c", "conv2d", 2, 4, 8, 32, 32, 3, 3, 1, 1, 1, 1), 2,
         Recipe("channel_lognormal", sigma=1.0)),
        (LayerShape("c", "conv2d", 3, 33, 40, 8, 8, 3, 3, 1, 1, 1, 1), 2,
         Recipe("channel_lognormal", sigma=1.0)),
    ]
    runs = []
    size = 0
    for i, (layer, bits, recipe) in enumerate(layers):
        fqt_, ref, desc, cfg, X, W, dY = _run_case(layer, bits, 0, recipe, "f32", data_seed=i)
        runs.append((layer, ref, desc, cfg, X, W, dY))
        size = max(size, fqt.fqt_workspace_size(desc, cfg, fqt.FQT_WS_LAYER))
    ws = torch.zeros(size, dtype=torch.uint8, device="cuda")
    state = fqt.FQT_WS_STATE_BYTES
    for rnd in range(2):
        for layer, ref, desc, cfg, X, W, dY in runs:
            _announce(f"[gpu parity] shared workspace round {rnd}: {layer}")
            dX, dW = torch.full_like(X, 7.0), torch.full_like(W, 7.0)
            fqt.fqt_layer_backward(desc, cfg, X, W, dY, dX, dW, ws)
            torch.cuda.synchronize()
            _assert_rescaled(dW, ref.dW, ref.dW_t1, ref.dW_t2, 1e-5, "dW")
            _assert_rescaled(dX, ref.dX, ref.dX_t1, ref.dX_t2, 1e-5, "dX")
            assert torch.count_nonzero(ws[:state]).item() == 0, "state bytes left non-zero"


FORWARD_CASES = [
    ("conv3x3_p1", LayerShape("c", "conv2d", 3, 7, 70, 9, 9, 3, 3, 1, 1, 1, 1), "f32"),
    ("conv_s2", LayerShape("c", "conv2d", 2, 16, 32, 11, 11, 3, 3, 2, 2, 1, 1), "f32"),
    ("conv1x1_s2", LayerShape("c", "conv2d", 4, 64, 128, 8, 8, 1, 1, 2, 2, 0, 0), "f32"),
    ("conv7x7_s2", LayerShape("c", "conv2d", 2, 3, 64, 32, 32, 7, 7, 2, 2, 3, 3), "f32"),
    ("conv5x5_p2", LayerShape("c", "conv2d", 3, 6, 40, 10, 10, 5, 5, 1, 1, 2, 2), "f32"),
    ("conv2x3_mixed", LayerShape("c", "conv2d", 2, 5, 9, 6, 7, 2, 3, 1, 2, 0, 1), "f32"),
    ("conv_p64_bf16", LayerShape("c", "conv2d", 5, 33, 96, 8, 8, 3, 3, 1, 1, 1, 1), "bf16"),
    ("linear_ragged", LayerShape("fc", "linear", 37, 300, 77), "f32"),
    ("linear_wide", LayerShape("fc", "linear", 64, 2048, 1000), "f32"),
    ("vgg_cifar_full", WORKLOADS["vgg_cifar_conv3x3_256"].layers[0], "f32"),
]


@pytest.mark.parametrize("name,layer,dtype", FORWARD_CASES, ids=[c[0] for c in FORWARD_CASES])
def test_forward_matches_oracle(name, layer, dtype):
    """fqt_binary_forward against the oracle's forward: the integer product bit-exact, Y
    within the one float32 rounding of gamma * I (bf16 Y: within bf16 rounding)."""
    _announce(f"[gpu parity] forward {name}: {layer} {dtype}")
    fqt = _fqt()
    x, w, _ = draw_layer(layer, Recipe(), 7, dtype)
    gamma = np.random.default_rng(11).standard_normal(layer.D).astype(np.float32)
    ref = ofqt.layer_forward(x, w, gamma, stride=layer.stride, pad=layer.pad)
    dt = fqt.FQT_BF16 if dtype == "bf16" else fqt.FQT_F32
    desc = fqt.layer_desc(layer, dy_dtype=dt, x_dtype=dt, w_dtype=fqt.FQT_F32, dx_dtype=dt)
    X, W = _to_dev(x, dtype), _to_dev(w, "f32")
    G = torch.from_numpy(gamma).cuda()
    ydt = torch.bfloat16 if dtype == "bf16" else torch.float32
    Y = torch.full(ref.Y.shape, 7.0, dtype=ydt, device="cuda")
    I = torch.full(ref.I.shape, 7, dtype=torch.int32, device="cuda")
    ws = fqt.workspace(desc, None, fqt.FQT_WS_FORWARD)
    for _ in range(2):                 # a reused workspace gives the same result
        fqt.fqt_binary_forward(desc, X, W, G, Y, I, ws)
        torch.cuda.synchronize()
        assert np.array_equal(I.cpu().numpy(), ref.I), "forward integer product"
        g = Y.float().cpu().numpy().astype(np.float64)
        rel = 2.0 ** -8 if dtype == "bf16" else 2.0 ** -24
        assert (np.abs(g - ref.Y) <= rel * np.abs(ref.Y)).all(), "forward output"


def test_garbage_workspace_after_init():
    """A layer workspace filled with garbage bytes, then prepared by fqt_workspace_init, gives
    the oracle's result; a second call on it (state left by the first) gives the same bits."""
    fqt = _fqt()
    layer = WORKLOADS["vgg_cifar_conv3x3_256"].layers[0]
    wl = WORKLOADS["vgg_cifar_conv3x3_256"]
    _announce("[gpu parity] garbage workspace + fqt_workspace_init")
    fqt_, ref, desc, cfg, X, W, dY = _run_case(layer, wl.bits, wl.agp_mode, wl.recipe, wl.dtype,
                                              seed=wl.philox_seed, step=0, layer_id=0,
                                              data_seed=wl.seed)
    n = fqt.fqt_workspace_size(desc, cfg, fqt.FQT_WS_LAYER)
    ws = torch.full((n,), 0xAB, dtype=torch.uint8, device="cuda")
    fqt.fqt_workspace_init(ws)
    dX, dW = torch.empty_like(X), torch.empty_like(W)
    outs = []
    for _ in range(2):
        fqt.fqt_layer_backward(desc, cfg, X, W, dY, dX, dW, ws)
        torch.cuda.synchronize()
        _assert_rescaled(dW, ref.dW, ref.dW_t1, ref.dW_t2, 1e-5, "dW")
        _assert_rescaled(dX, ref.dX, ref.dX_t1, ref.dX_t2, 1e-5, "dX")
        outs.append((dX.clone(), dW.clone()))
    assert torch.equal(outs[0][0], outs[1][0]) and torch.equal(outs[0][1], outs[1][1])
    assert torch.count_nonzero(ws[:fqt.FQT_WS_STATE_BYTES]).item() == 0
