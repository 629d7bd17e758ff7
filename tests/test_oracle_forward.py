"""Pins of the oracle's binary forward (Section 5.1; Appendix C, Alg. 1 forward and the
Unfolder): a torch float64 convolution of the sign tensors, brute-force loops, the linear
special case, a closed form at the borders, and planted mistakes that the pins catch."""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import fqt
from paper_2408_14267_amd.workloads import LayerShape, Recipe, draw_layer

LAYERS = [
    LayerShape("lin", "linear", 7, 13, 5),
    LayerShape("c3", "conv2d", 3, 4, 5, 5, 6, 3, 3, 1, 1, 1, 1),
    LayerShape("c3s2", "conv2d", 2, 3, 4, 7, 5, 3, 3, 2, 2, 1, 1),
    LayerShape("c1s2", "conv2d", 3, 5, 6, 4, 4, 1, 1, 2, 2, 0, 0),
    LayerShape("c2x3", "conv2d", 2, 3, 3, 5, 6, 2, 3, 1, 2, 0, 1),
    LayerShape("c5p2", "conv2d", 2, 2, 3, 6, 6, 5, 5, 1, 1, 2, 2),
]


def _signs(a):
    return np.where(np.asarray(a) > 0, 1.0, -1.0)


def _torch_forward(x, w, layer):
    """sign(X) padded with -1 (the padding reading), convolved in float64 with sign(W)."""
    if layer.kind == "linear":
        return _signs(x) @ _signs(w).T
    sx = torch.from_numpy(_signs(x))
    sx = F.pad(sx, (layer.pw, layer.pw, layer.ph, layer.ph), value=-1.0)
    return F.conv2d(sx, torch.from_numpy(_signs(w)), stride=layer.stride).numpy()


def _gamma(layer, seed=3):
    return np.random.default_rng(seed).standard_normal(layer.D)


@pytest.mark.parametrize("layer", LAYERS, ids=lambda l: l.name)
def test_forward_matches_torch_sign_convolution(layer):
    x, w, _ = draw_layer(layer, Recipe(), 0)
    g = _gamma(layer)
    f = fqt.layer_forward(x, w, g, layer.stride, layer.pad)
    ref = _torch_forward(x, w, layer)
    assert np.array_equal(f.I, np.rint(ref).astype(np.int64))
    shape = (1, -1) if layer.kind == "linear" else (1, -1, 1, 1)
    np.testing.assert_array_equal(f.Y, ref * g.reshape(shape))


def test_forward_brute_force_loops():
    layer = LayerShape("c", "conv2d", 2, 3, 2, 5, 4, 2, 3, 2, 1, 1, 1)
    x, w, _ = draw_layer(layer, Recipe(), 5)
    sx, sw = _signs(x), _signs(w)
    N, C, H, W = x.shape
    D, _, kh, kw = w.shape
    (sh, sw_), (ph, pw) = layer.stride, layer.pad
    Ho, Wo = (H + 2 * ph - kh) // sh + 1, (W + 2 * pw - kw) // sw_ + 1
    want = np.zeros((N, D, Ho, Wo), dtype=np.int64)
    for n in range(N):
        for d in range(D):
            for ho in range(Ho):
                for wo in range(Wo):
                    acc = 0
                    for c in range(C):
                        for i in range(kh):
                            for j in range(kw):
                                h, v = ho * sh - ph + i, wo * sw_ - pw + j
                                s = sx[n, c, h, v] if 0 <= h < H and 0 <= v < W else -1.0
                                acc += int(s * sw[d, c, i, j])
                    want[n, d, ho, wo] = acc
    got = fqt.layer_forward(x, w, np.ones(D), layer.stride, layer.pad)
    assert np.array_equal(got.I, want)


def test_forward_all_positive_closed_form():
    """All-positive X and W: a window counts +1 per in-image tap and -1 per padded tap, so
    I = C (kh kw - 2 * padded taps); the 3x3 pad-1 corner has 5 padded taps: I = -C."""
    N, C, H, W, D = 2, 3, 4, 5, 2
    x = np.ones((N, C, H, W), np.float32)
    w = np.ones((D, C, 3, 3), np.float32)
    f = fqt.layer_forward(x, w, np.array([1.0, -2.0]), (1, 1), (1, 1))
    assert (f.I[:, :, 1:-1, 1:-1] == 9 * C).all()
    assert (f.I[:, :, 0, 0] == -C).all() and (f.I[:, :, -1, -1] == -C).all()
    assert (f.I[:, :, 0, 2] == 3 * C).all()            # top edge: 3 padded taps
    np.testing.assert_array_equal(f.Y[:, 1], -2.0 * f.I[:, 1])


def test_forward_sign_of_zero_is_minus_one():
    x = np.zeros((1, 2), np.float32)
    w = np.array([[1.0, 1.0], [-1.0, 0.0]], np.float32)
    f = fqt.layer_forward(x, w, np.ones(2))
    assert f.I.tolist() == [[-2, 2]]           # sign(0) = -1 in X and in W


def test_planted_forward_mistakes_are_caught():
    """Two plausible mistakes, written here as variants of the oracle, disagree with the
    torch pin: padding with sign +1 and a weight operand transposed within the kernel."""
    layer = LAYERS[1]
    x, w, _ = draw_layer(layer, Recipe(), 1)
    ref = np.rint(_torch_forward(x, w, layer)).astype(np.int64)
    # +1 padding: binarize, pad with ones, convolve.
    sx = F.pad(torch.from_numpy(_signs(x)), (1, 1, 1, 1), value=1.0)
    plus_pad = F.conv2d(sx, torch.from_numpy(_signs(w))).numpy()
    assert not np.array_equal(np.rint(plus_pad).astype(np.int64), ref)
    # kernel window transposed (i <-> j) in the weight operand.
    wt = np.ascontiguousarray(np.swapaxes(w, 2, 3))
    assert not np.array_equal(fqt.layer_forward(x, wt, np.ones(layer.D), (1, 1), (1, 1)).I, ref)
