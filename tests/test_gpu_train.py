"""The training wrapper (binary layers as torch modules over the C ABI) against the oracle:
the forward output, dX, dW and dGamma of one binary layer, and a few whole training steps
of the binary VGG-16 and ResNet-18."""
import sys

import numpy as np
import pytest

from oracle import fqt as ofqt
from paper_2408_14267_amd.workloads import LayerShape, Recipe, draw_layer

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def _announce(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.mark.parametrize("kind", ["conv", "linear"])
def test_binary_layer_module_matches_oracle(kind):
    from paper_2408_14267_amd import fqt, train
    _announce(f"[gpu train] binary {kind} module")
    if kind == "conv":
        L = LayerShape("c", "conv2d", 6, 8, 24, 7, 7, 3, 3, 1, 1, 1, 1)
        mod = train.BinaryConv2d(8, 24, 3, 1, 1, bits=2, layer_id=3, seed=9).cuda()
    else:
        L = LayerShape("fc", "linear", 16, 40, 24)
        mod = train.BinaryLinear(40, 24, bits=2, layer_id=3, seed=9).cuda()
    x, w, dy = draw_layer(L, Recipe("sample_lognormal", sigma=1.0), 4)
    gamma = np.random.default_rng(2).uniform(0.5, 1.5, L.D).astype(np.float32)
    with torch.no_grad():
        mod.weight.copy_(torch.from_numpy(w))
        mod.gamma.copy_(torch.from_numpy(gamma))
    X = torch.from_numpy(x).cuda().requires_grad_(True)
    Y = mod(X)
    fref = ofqt.layer_forward(x, w, gamma, stride=L.stride, pad=L.pad)
    got = Y.detach().cpu().numpy().astype(np.float64)
    assert (np.abs(got - fref.Y) <= 2.0 ** -24 * np.abs(fref.Y)).all(), "forward"
    Y.backward(torch.from_numpy(dy).cuda())
    torch.cuda.synchronize()
    # The library quantizes the gradient of the binary product, dy * Gamma (one float32
    # product per element, the same on both sides), with step 0 of this layer's stream.
    shape = (1, -1) + (1,) * (dy.ndim - 2)
    g = (dy * gamma.reshape(shape)).astype(np.float32)
    bref = ofqt.layer_backward(x, w, g, 2, ofqt.AGP_BERNOULLI, seed=9, step=0, layer_id=3,
                               stride=L.stride, pad=L.pad)
    mask = np.abs(x) <= 1
    dx = X.grad.cpu().numpy().astype(np.float64)
    assert (np.abs(dx - bref.dX * mask) <= 1e-5 * (np.abs(bref.dX_t1) + np.abs(bref.dX_t2)) + 1e-30).all()
    dw = mod.weight.grad.cpu().numpy().astype(np.float64)
    assert (np.abs(dw - bref.dW) <= 1e-5 * (np.abs(bref.dW_t1) + np.abs(bref.dW_t2)) + 1e-30).all()
    dg_ref = (dy.astype(np.float64) * fref.I).sum(axis=(0,) + tuple(range(2, dy.ndim)))
    np.testing.assert_allclose(mod.gamma.grad.cpu().numpy(), dg_ref, rtol=1e-5,
                               atol=1e-6 * np.abs(dy).sum())
    assert mod.step == 1


@pytest.mark.parametrize("net", ["vgg16", "resnet18"])
def test_binary_network_training_steps(net):
    """Three Adam steps of the binary network on a fixed random batch: finite losses, every
    binary layer's latent weights and Gamma move, and the library's step counter advances."""
    from paper_2408_14267_amd import train
    _announce(f"[gpu train] {net} steps")
    torch.manual_seed(0)
    model = (train.VGG16(10, 32, binary=True, bits=4, fc=512) if net == "vgg16"
             else train.ResNet18(10, binary=True, bits=4)).cuda()
    opt = torch.optim.Adam(model.parameters(), lr=1e-3)
    x = torch.randn(16, 3, 32, 32, device="cuda")
    y = torch.randint(0, 10, (16,), device="cuda")
    binary = [m for m in model.modules() if isinstance(m, train._BinaryBase)]
    before = [m.weight.detach().clone() for m in binary]
    losses = [float(train.train_step(model, opt, x, y).detach()) for _ in range(3)]
    torch.cuda.synchronize()
    assert all(np.isfinite(losses)), losses
    for m, w0 in zip(binary, before):
        assert not torch.equal(m.weight.detach(), w0)
        assert m.step == 3
