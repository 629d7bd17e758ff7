"""Host-side checks of the C ABI: the library loads, exports what include/fqt.h declares,
and validates arguments before launching anything (no GPU needed)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "fqt.h")

fqt = pytest.importorskip("paper_2408_14267_amd.fqt", reason="libfqt.so not built")

from paper_2408_14267_amd.workloads import LayerShape, WORKLOADS  # noqa: E402


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^(?:int|const char \*)\s*(fqt_\w+)\(", text, flags=re.M)))


def test_exports_every_declared_symbol():
    names = declared_functions()
    assert len(names) == 15
    lib = ctypes.CDLL(fqt.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n
    assert sorted(fqt.EXPORTED) == names


def test_status_strings():
    for s in range(-7, 1):
        assert fqt.fqt_status_string(s).startswith("FQT_")
    assert "unknown" in fqt.fqt_status_string(5)


def _desc(**kw):
    L = WORKLOADS["vgg_cifar_conv3x3_256"].layers[0]
    d = fqt.layer_desc(L)
    for k, v in kw.items():
        setattr(d, k, v)
    return d


@pytest.mark.parametrize("field,value,status", [
    ("kind", 7, fqt.FQT_E_INVAL), ("dy_dtype", 3, fqt.FQT_E_DTYPE), ("N", 0, fqt.FQT_E_SHAPE),
    ("D", -1, fqt.FQT_E_SHAPE), ("kh", 0, fqt.FQT_E_SHAPE), ("sh", 0, fqt.FQT_E_SHAPE),
    ("ph", -1, fqt.FQT_E_SHAPE), ("kh", 11, fqt.FQT_E_SHAPE), ("N", 16385, fqt.FQT_E_SHAPE),
    ("D", 20000, fqt.FQT_E_SHAPE)])
def test_descriptor_validation(field, value, status):
    with pytest.raises(fqt.FqtError) as e:
        fqt.fqt_workspace_size(_desc(**{field: value}), fqt.quant_cfg(4))
    assert e.value.status == status


def test_linear_geometry_must_be_trivial():
    d = fqt.layer_desc(LayerShape("fc", "linear", 8, 16, 4))
    d.kh = 3
    with pytest.raises(fqt.FqtError) as e:
        fqt.fqt_workspace_size(d, fqt.quant_cfg(2))
    assert e.value.status == fqt.FQT_E_SHAPE


@pytest.mark.parametrize("bits,mode", [(0, 0), (9, 0), (2, 3), (2, -1)])
def test_cfg_validation(bits, mode):
    with pytest.raises(fqt.FqtError) as e:
        fqt.fqt_workspace_size(_desc(), fqt.quant_cfg(bits, mode))
    assert e.value.status == fqt.FQT_E_INVAL


def test_workspace_and_plane_sizes():
    d = _desc()
    c = fqt.quant_cfg(4)
    psq, pcq, psq_b, pcq_b = fqt.fqt_qgrad_words(d, c)
    R = 128 * 64
    assert psq == 4 * R * 4 and pcq == 4 * 256 * (R // 64)
    assert psq_b == R * 256 and pcq_b == 256 * R
    ws_layer = fqt.fqt_workspace_size(d, c, fqt.FQT_WS_LAYER)
    ws_q = fqt.fqt_workspace_size(d, c, fqt.FQT_WS_QUANTIZE)
    assert ws_layer > (psq + pcq) * 8 > ws_q > 0
    with pytest.raises(fqt.FqtError):
        fqt.fqt_workspace_size(d, c, 7)


def test_null_and_small_workspace_rejected_before_launch():
    lib = fqt._lib
    d = _desc()
    c = fqt.quant_cfg(4)
    fake = ctypes.c_void_p(1 << 20)          # never dereferenced: validation fails first
    st = lib.fqt_layer_backward(ctypes.byref(d), ctypes.byref(c), None, fake, fake, fake, fake,
                                fake, 1 << 30, None)
    assert st == fqt.FQT_E_NULL
    st = lib.fqt_layer_backward(ctypes.byref(d), ctypes.byref(c), fake, fake, fake, fake, fake,
                                fake, 16, None)
    assert st == fqt.FQT_E_WORKSPACE
    mis = ctypes.c_void_p((1 << 20) + 4)
    st = lib.fqt_layer_backward(ctypes.byref(d), ctypes.byref(c), fake, fake, mis, fake, fake,
                                fake, 1 << 30, None)
    assert st == fqt.FQT_E_ALIGN
    st = lib.fqt_pack_bits(fake, 0, 10, 10, 5, fqt.FQT_PACK_ALONG_COLS, None, fake, None, None)
    assert st == fqt.FQT_E_SHAPE
    st = lib.fqt_pack_bits(fake, 0, 10, 10, 10, 5, None, fake, None, None)
    assert st == fqt.FQT_E_INVAL
    st = lib.fqt_pack_bits(fake, 0, 0, 0, 0, fqt.FQT_PACK_IM2COL, None, fake, None, None)
    assert st == fqt.FQT_E_NULL
    q = fqt.fqt_qgrad()
    st = lib.fqt_binary_gemm_dw(ctypes.byref(d), ctypes.byref(c), ctypes.byref(q), fake, fake,
                                None, fake, 1 << 30, None)
    assert st == fqt.FQT_E_NULL
    st = lib.fqt_pack_weight_signs(ctypes.byref(d), fake, fake, None, None)
    assert st == fqt.FQT_E_NULL
    st = lib.fqt_pack_weight_signs(ctypes.byref(d), fake, ctypes.c_void_p((1 << 20) + 8), fake,
                                   None)
    assert st == fqt.FQT_E_ALIGN            # the sign bytes must be 16-byte aligned


def test_state_bytes_constant_matches_header():
    text = open(HEADER).read()
    m = re.search(r"#define FQT_WS_STATE_BYTES (\d+)", text)
    assert m and int(m.group(1)) == fqt.FQT_WS_STATE_BYTES
    m = re.search(r"#define FQT_NOALLOC_SCRATCH_BYTES \((\d+)u << (\d+)\)", text)
    assert m and int(m.group(1)) << int(m.group(2)) == fqt.FQT_NOALLOC_SCRATCH_BYTES
    d = _desc()
    c = fqt.quant_cfg(4)
    assert fqt.fqt_workspace_size(d, c, fqt.FQT_WS_QUANTIZE) > fqt.FQT_WS_STATE_BYTES


def test_forward_workspace_and_validation():
    lib = fqt._lib
    d = _desc()
    n = fqt.fqt_workspace_size(d, None, fqt.FQT_WS_FORWARD)     # no quantizer config needed
    L = WORKLOADS["vgg_cifar_conv3x3_256"].layers[0]
    K, R = L.C * 9, L.N * 64
    assert n >= K * (R // 64) * 8 * 2 + 256 * K
    fake = ctypes.c_void_p(1 << 20)
    st = lib.fqt_binary_forward(ctypes.byref(d), fake, fake, None, fake, None, fake, n, None)
    assert st == fqt.FQT_E_NULL
    st = lib.fqt_binary_forward(ctypes.byref(d), fake, fake, fake, fake, None, fake, 16, None)
    assert st == fqt.FQT_E_WORKSPACE
    st = lib.fqt_binary_forward(ctypes.byref(d), fake, fake, ctypes.c_void_p((1 << 20) + 2),
                                fake, None, fake, n, None)
    assert st == fqt.FQT_E_ALIGN


def test_workspace_init_validation():
    lib = fqt._lib
    fake = ctypes.c_void_p(1 << 20)          # never dereferenced: validation fails first
    assert lib.fqt_workspace_init(None, 1 << 20, None) == fqt.FQT_E_NULL
    assert lib.fqt_workspace_init(ctypes.c_void_p((1 << 20) + 16), 1 << 20, None) == fqt.FQT_E_ALIGN
    assert lib.fqt_workspace_init(fake, fqt.FQT_WS_STATE_BYTES - 1, None) == fqt.FQT_E_WORKSPACE


@pytest.mark.parametrize("bits,n,h,ok", [(8, 128, 65793, True), (8, 5, 1684301, False),
                                         (7, 8, 2113665, True), (7, 11, 1537211, False)])
def test_dw_integer_range_rejected_before_launch(bits, n, h, ok):
    """The dW integer I = sum_r q s reaches (2^b - 1) * N*Ho*Wo; layers where that exceeds
    2^31 - 1 are refused (FQT_E_SHAPE) by the dW product and the layer backward, before any
    launch; the quantizer alone still accepts them.  The rows N*Ho*Wo sit on either side of
    floor((2^31 - 1) / (2^b - 1)): 8421504 / 8421505 for b = 8, 16909320 / 16909321 for
    b = 7 (1x1 convolutions over h x 1 maps; b <= 6 cannot reach the bound within the
    code-array size limit)."""
    lib = fqt._lib
    d = fqt.layer_desc(LayerShape("c", "conv2d", n, 1, 1, h, 1))
    R = n * h
    assert (((1 << bits) - 1) * R <= (1 << 31) - 1) == ok
    c = fqt.quant_cfg(bits, fqt.FQT_AGP_OFF)
    fake = ctypes.c_void_p(1 << 20)
    q = fqt.fqt_qgrad(*([1 << 20] * 14))
    st_dw = lib.fqt_binary_gemm_dw(ctypes.byref(d), ctypes.byref(c), ctypes.byref(q), fake,
                                   fake, None, fake, 0, None)
    st_layer = lib.fqt_layer_backward(ctypes.byref(d), ctypes.byref(c), fake, fake, fake, fake,
                                      fake, fake, 0, None)
    if ok:       # past the range check: the zero-byte workspace is what fails
        assert st_dw == fqt.FQT_E_WORKSPACE and st_layer == fqt.FQT_E_WORKSPACE
    else:
        assert st_dw == fqt.FQT_E_SHAPE and st_layer == fqt.FQT_E_SHAPE
    fqt.fqt_workspace_size(d, c, fqt.FQT_WS_QUANTIZE)       # the quantizer has no such bound


def test_noalloc_rejects_layers_beyond_its_scratch_before_launch():
    """fqt_layer_backward_noalloc validates like fqt_layer_backward and refuses a layer whose
    workspace exceeds the static scratch (VGG-16 conv2 at batch 64 needs 742 MiB) with
    FQT_E_WORKSPACE, before it touches the device."""
    lib = fqt._lib
    fake = ctypes.c_void_p(1 << 20)
    vgg = {L.name: L for L in WORKLOADS["vgg16_224_bf16"].layers}
    d = fqt.layer_desc(vgg["conv2"], fqt.FQT_BF16, fqt.FQT_BF16, fqt.FQT_F32, fqt.FQT_BF16)
    c = fqt.quant_cfg(2)
    assert fqt.fqt_workspace_size(d, c) > fqt.FQT_NOALLOC_SCRATCH_BYTES
    st = lib.fqt_layer_backward_noalloc(ctypes.byref(d), ctypes.byref(c), fake, fake, fake,
                                        fake, fake, None)
    assert st == fqt.FQT_E_WORKSPACE
    d2 = _desc()
    assert fqt.fqt_workspace_size(d2, fqt.quant_cfg(4)) <= fqt.FQT_NOALLOC_SCRATCH_BYTES
    st = lib.fqt_layer_backward_noalloc(ctypes.byref(d2), ctypes.byref(c), None, fake, fake,
                                        fake, fake, None)
    assert st == fqt.FQT_E_NULL
    st = lib.fqt_layer_backward_noalloc(ctypes.byref(d2), ctypes.byref(c), fake, fake,
                                        ctypes.c_void_p((1 << 20) + 4), fake, fake, None)
    assert st == fqt.FQT_E_ALIGN


def test_binding_sizes_follow_the_descriptor():
    # 3x3 conv 256 -> 256 on 8x8, N = 128: R = 8192 rows, K = 2304 lines, Wd = 4 words of D.
    z = fqt._sizes(_desc())
    assert z == {"X": 128 * 256 * 64, "W": 256 * 2304, "dY": 128 * 256 * 64,
                 "xsign": 128 * 2304, "wsign": 2304 * 64 * 4, "K": 2304}
    lin = fqt._sizes(fqt.layer_desc(LayerShape("fc", "linear", 32, 256, 128)))
    assert lin == {"X": 32 * 256, "W": 128 * 256, "dY": 32 * 128, "xsign": 256,
                   "wsign": 256 * 128, "K": 256}
    # Strided, padded conv: Ho = Wo = (9 + 2 - 3) // 2 + 1 = 5.
    st = fqt._sizes(fqt.layer_desc(LayerShape("c", "conv2d", 2, 3, 5, 9, 9, 3, 3, 2, 2, 1, 1)))
    assert st["dY"] == 2 * 5 * 25 and st["xsign"] == 1 * 27 and st["X"] == 2 * 3 * 81


def test_binding_rejects_mismatched_tensors_before_launch():
    torch = pytest.importorskip("torch")
    L = WORKLOADS["vgg_cifar_conv3x3_256"].layers[0]
    d = fqt.layer_desc(L, fqt.FQT_BF16, fqt.FQT_BF16, fqt.FQT_F32, fqt.FQT_BF16)
    c = fqt.quant_cfg(4)
    z = fqt._sizes(d)
    X = torch.empty(z["X"], dtype=torch.bfloat16)
    W = torch.empty(z["W"], dtype=torch.float32)
    dY = torch.empty(z["dY"], dtype=torch.bfloat16)
    dW = torch.empty(z["W"], dtype=torch.float32)
    ws = torch.empty(16, dtype=torch.uint8)
    # A float32 X against a bf16 descriptor (the kernels would read twice its bytes).
    with pytest.raises(ValueError, match="dtype"):
        fqt.fqt_layer_backward(d, c, X.float(), W, dY, X, dW, ws)
    with pytest.raises(ValueError, match="elements"):
        fqt.fqt_layer_backward(d, c, X, W, dY[:-1], X, dW, ws)
    with pytest.raises(ValueError, match="contiguous"):
        fqt.fqt_pack_input_signs(d, X.view(2, -1).t(), torch.empty(z["xsign"], dtype=torch.int64))
    with pytest.raises(ValueError, match="elements"):
        fqt.fqt_pack_weight_signs(d, W, torch.empty(z["wsign"] - 1, dtype=torch.int8),
                                  torch.empty(z["K"], dtype=torch.int32))
    # Everything the descriptor asks for, but host memory: still refused, nothing launched.
    with pytest.raises(ValueError, match="device tensor"):
        fqt.fqt_layer_backward(d, c, X, W, dY, X, dW, ws)
