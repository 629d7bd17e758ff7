"""Training with binary layers under 1-bit FQT: torch modules over the C ABI.

BinaryConv2d / BinaryLinear compute the binary forward of Section 5.1,
H = (sign(X) sign(W)) * Gamma with a learnable per-output-channel Gamma, through
fqt_binary_forward, and their backward through fqt_layer_backward: AGP + SCQ
quantization of the gradient of the binary product, the two binary products and
the rescale (Sections 5.2, 5.3; Appendix C, Alg. 1).  Around those two calls the
autograd function applies what the paper leaves to the training loop:

  * the gradient of the binary product is dL/dH * Gamma (per output channel), the
    chain rule through H = I * Gamma; it is the tensor the library quantizes;
  * dGamma_d = sum over samples and pixels of dL/dH * I (I = the integer product,
    kept from the forward);
  * the straight-through estimator for the sign binarizer (Section 3.1): dL/dX =
    dL/dsign(X) where |X| <= 1, 0 elsewhere; the latent weights take dL/dsign(W)
    unchanged.

Adam (Section 4.1) updates the latent weights.  Networks follow the paper's setup
(Section 6 and Appendix D): the first and last layers, the 1x1 shortcuts of
ResNet, batch norm and the activations stay in float32; every other convolution
and fully connected layer is binary.
"""
import torch
import torch.nn as nn
import torch.nn.functional as F

from . import fqt


class _BinaryLayerFn(torch.autograd.Function):
    @staticmethod
    def forward(ctx, x, w, gamma, layer):
        desc = layer.desc(x.shape)
        y = torch.empty(layer.y_shape(x.shape), dtype=torch.float32, device=x.device)
        i = torch.empty(y.shape, dtype=torch.int32, device=x.device)
        fqt.fqt_binary_forward(desc, x, w, gamma, y, i, layer.ws_forward(desc))
        ctx.save_for_backward(x, w, gamma, i)
        ctx.layer = layer
        return y

    @staticmethod
    def backward(ctx, dy):
        x, w, gamma, i = ctx.saved_tensors
        layer = ctx.layer
        shape = (1, -1) + (1,) * (dy.dim() - 2)
        g = (dy * gamma.view(shape)).contiguous()          # gradient of the binary product
        dx = torch.empty_like(x)
        dw = torch.empty_like(w)
        desc = layer.desc(x.shape)
        cfg = fqt.quant_cfg(layer.bits, layer.agp_mode, layer.seed, layer.step, layer.layer_id)
        fqt.fqt_layer_backward(desc, cfg, x, w, g, dx, dw, layer.ws_backward(desc, cfg))
        layer.step += 1
        dx = dx * (x.abs() <= 1)                            # straight-through estimator
        dims = [0] + list(range(2, dy.dim()))
        dgamma = (dy * i.to(torch.float32)).sum(dim=dims)
        return dx, dw, dgamma, None


class _BinaryBase(nn.Module):
    """Latent float32 weight, Gamma, quantizer settings and per-shape workspaces."""

    def __init__(self, weight_shape, out_features, bits, agp_mode, layer_id, seed):
        super().__init__()
        self.weight = nn.Parameter(torch.empty(weight_shape))
        nn.init.kaiming_uniform_(self.weight, a=5 ** 0.5)
        self.gamma = nn.Parameter(torch.full((out_features,), 1.0 / (self.weight[0].numel() ** 0.5)))
        self.bits, self.agp_mode, self.layer_id, self.seed = bits, agp_mode, layer_id, seed
        self.step = 0
        self._ws = {}

    def _workspace(self, key, desc, cfg, which):
        ws = self._ws.get(key)
        if ws is None:
            ws = fqt.workspace(desc, cfg, which, device=self.weight.device)
            self._ws[key] = ws
        return ws

    def ws_forward(self, desc):
        return self._workspace(("f", desc.N, desc.H, desc.W), desc, None, fqt.FQT_WS_FORWARD)

    def ws_backward(self, desc, cfg):
        return self._workspace(("b", desc.N, desc.H, desc.W), desc, cfg, fqt.FQT_WS_LAYER)

    def forward(self, x):
        return _BinaryLayerFn.apply(x.contiguous(), self.weight, self.gamma, self)


class BinaryConv2d(_BinaryBase):
    def __init__(self, cin, cout, k, stride=1, padding=0, bits=4, agp_mode=fqt.FQT_AGP_BERNOULLI,
                 layer_id=0, seed=0):
        super().__init__((cout, cin, k, k), cout, bits, agp_mode, layer_id, seed)
        self.cin, self.cout, self.k, self.stride, self.padding = cin, cout, k, stride, padding

    def y_shape(self, xs):
        return (xs[0], self.cout, (xs[2] + 2 * self.padding - self.k) // self.stride + 1,
                (xs[3] + 2 * self.padding - self.k) // self.stride + 1)

    def desc(self, xs):
        return fqt.fqt_layer_desc(fqt.FQT_CONV2D, fqt.FQT_F32, fqt.FQT_F32, fqt.FQT_F32, fqt.FQT_F32,
                                  xs[0], self.cin, xs[2], xs[3], self.cout, self.k, self.k,
                                  self.stride, self.stride, self.padding, self.padding)


class BinaryLinear(_BinaryBase):
    def __init__(self, fin, fout, bits=4, agp_mode=fqt.FQT_AGP_BERNOULLI, layer_id=0, seed=0):
        super().__init__((fout, fin), fout, bits, agp_mode, layer_id, seed)
        self.fin, self.fout = fin, fout

    def y_shape(self, xs):
        return (xs[0], self.fout)

    def desc(self, xs):
        return fqt.fqt_layer_desc(fqt.FQT_LINEAR, fqt.FQT_F32, fqt.FQT_F32, fqt.FQT_F32, fqt.FQT_F32,
                                  xs[0], self.fin, 1, 1, self.fout, 1, 1, 1, 1, 0, 0)


# ----------------------------------------------------------------------------- networks

_VGG16 = [64, 64, "M", 128, 128, "M", 256, 256, 256, "M", 512, 512, 512, "M", 512, 512, 512, "M"]


class VGG16(nn.Module):
    """VGG-16 with batch norm: 13 3x3 convolutions, five max-pools, fc6 / fc7 / fc8.  With
    binary=True every convolution but the first, and fc6 / fc7, are binary layers; the
    first convolution and fc8 stay float32 (binary=False: all float32, for comparison)."""

    def __init__(self, num_classes=10, res=32, binary=True, bits=4, fc=4096):
        super().__init__()
        layers, cin, lid = [], 3, 0
        for v in _VGG16:
            if v == "M":
                layers.append(nn.MaxPool2d(2))
                continue
            if binary and cin != 3:
                layers.append(BinaryConv2d(cin, v, 3, 1, 1, bits=bits, layer_id=lid))
            else:
                layers.append(nn.Conv2d(cin, v, 3, 1, 1, bias=False))
            layers += [nn.BatchNorm2d(v), nn.Hardtanh() if binary else nn.ReLU()]
            cin, lid = v, lid + 1
        self.features = nn.Sequential(*layers)
        flat = 512 * (res // 32) ** 2
        lin = (lambda i, o, l: BinaryLinear(i, o, bits=bits, layer_id=l)) if binary else \
            (lambda i, o, l: nn.Linear(i, o, bias=False))
        self.classifier = nn.Sequential(
            lin(flat, fc, 13), nn.BatchNorm1d(fc), nn.Hardtanh() if binary else nn.ReLU(),
            lin(fc, fc, 14), nn.BatchNorm1d(fc), nn.Hardtanh() if binary else nn.ReLU(),
            nn.Linear(fc, num_classes))

    def forward(self, x):
        return self.classifier(torch.flatten(self.features(x), 1))


class _Block(nn.Module):
    def __init__(self, cin, cout, stride, binary, bits, lid):
        super().__init__()
        conv = (lambda i, o, s, l: BinaryConv2d(i, o, 3, s, 1, bits=bits, layer_id=l)) if binary \
            else (lambda i, o, s, l: nn.Conv2d(i, o, 3, s, 1, bias=False))
        self.c1, self.b1 = conv(cin, cout, stride, lid), nn.BatchNorm2d(cout)
        self.c2, self.b2 = conv(cout, cout, 1, lid + 1), nn.BatchNorm2d(cout)
        self.act = nn.Hardtanh() if binary else nn.ReLU()
        self.down = None
        if stride != 1 or cin != cout:      # 1x1 shortcut projections stay float32
            self.down = nn.Sequential(nn.Conv2d(cin, cout, 1, stride, bias=False),
                                      nn.BatchNorm2d(cout))

    def forward(self, x):
        y = self.act(self.b1(self.c1(x)))
        y = self.b2(self.c2(y))
        return self.act(y + (x if self.down is None else self.down(x)))


class ResNet18(nn.Module):
    """ResNet-18 with the ImageNet stem (7x7/2 conv, 3x3/2 max-pool).  With binary=True the
    16 3x3 convolutions of the residual blocks are binary; the stem, the 1x1 shortcuts and
    the fc stay float32."""

    def __init__(self, num_classes=10, binary=True, bits=4):
        super().__init__()
        self.stem = nn.Sequential(nn.Conv2d(3, 64, 7, 2, 3, bias=False), nn.BatchNorm2d(64),
                                  nn.ReLU(), nn.MaxPool2d(3, 2, 1))
        blocks, cin, lid = [], 64, 1
        for stage, c in enumerate((64, 128, 256, 512)):
            for blk in range(2):
                s = 2 if stage > 0 and blk == 0 else 1
                blocks.append(_Block(cin, c, s, binary, bits, lid))
                cin, lid = c, lid + 2
        self.blocks = nn.Sequential(*blocks)
        self.fc = nn.Linear(512, num_classes)

    def forward(self, x):
        x = self.blocks(self.stem(x))
        return self.fc(torch.flatten(F.adaptive_avg_pool2d(x, 1), 1))


def train_step(model, opt, x, y, autocast_dtype=None):
    """One step: forward, cross-entropy loss, backward, Adam update.  Returns the loss."""
    opt.zero_grad(set_to_none=True)
    if autocast_dtype is not None:
        with torch.autocast("cuda", dtype=autocast_dtype):
            loss = F.cross_entropy(model(x), y)
    else:
        loss = F.cross_entropy(model(x), y)
    loss.backward()
    opt.step()
    return loss
