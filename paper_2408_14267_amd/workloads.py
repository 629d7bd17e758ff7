"""Seeded synthetic workloads for the 1-bit FQT layer backward.

Shapes and value distributions only -- none of the method's arithmetic lives
here.  Both the HIP path (tests, bench) and the CPU oracle are fed from these
generators.  Every tensor is drawn with numpy's ``default_rng(seed)`` in the
order x, w, dy (then any extra draws of dy's recipe), as float32; a bf16
workload rounds the float32 draws to bfloat16 (round to nearest even), so the
same values feed both sides exactly.

Recipes stand in for the paper's gradients, whose group ranges are highly
uneven across samples and channels (Section 5.2 and Appendix D.1 of the
paper); the datasets and trained models the paper measured are not used.
"""
from dataclasses import dataclass, field

import numpy as np


@dataclass(frozen=True)
class LayerShape:
    """A linear layer ([N][C] -> [N][D]) or a 2-D convolution (NCHW, weight [D][C][kh][kw])."""
    name: str
    kind: str                      # "linear" | "conv2d"
    N: int
    C: int
    D: int
    H: int = 1
    W: int = 1
    kh: int = 1
    kw: int = 1
    sh: int = 1
    sw: int = 1
    ph: int = 0
    pw: int = 0

    @property
    def Ho(self):
        return (self.H + 2 * self.ph - self.kh) // self.sh + 1

    @property
    def Wo(self):
        return (self.W + 2 * self.pw - self.kw) // self.sw + 1

    @property
    def x_shape(self):
        return (self.N, self.C) if self.kind == "linear" else (self.N, self.C, self.H, self.W)

    @property
    def w_shape(self):
        return (self.D, self.C) if self.kind == "linear" else (self.D, self.C, self.kh, self.kw)

    @property
    def dy_shape(self):
        return (self.N, self.D) if self.kind == "linear" else (self.N, self.D, self.Ho, self.Wo)

    @property
    def stride(self):
        return (self.sh, self.sw)

    @property
    def pad(self):
        return (self.ph, self.pw)

    def binary_macs(self):
        """Multiply-accumulates of one full-precision product of this layer's backward
        (dW and dX each take D * C*kh*kw * N*Ho*Wo)."""
        return self.D * self.C * self.kh * self.kw * self.N * self.Ho * self.Wo


@dataclass(frozen=True)
class Recipe:
    """How dy is drawn.  kind:
    "sample_lognormal"  dy = z * s_n, z ~ N(0,1), s_n ~ exp(sigma N(0,1)) per sample;
                        optionally `outlier_count` samples chosen without replacement
                        are multiplied by `outlier_factor`.
    "channel_lognormal" dy = z * s_d, s_d ~ exp(sigma N(0,1)) per output channel.
    "student_t"         dy ~ Student-t with `df` degrees of freedom, i.i.d.
    "sample_geometric"  dy = z * ratio^n for sample n (group ranges decaying geometrically).
    """
    kind: str = "sample_lognormal"
    sigma: float = 1.5
    outlier_count: int = 0
    outlier_factor: float = 100.0
    df: float = 3.0
    ratio: float = 0.8


@dataclass(frozen=True)
class Workload:
    name: str
    layers: tuple
    recipe: Recipe
    bits: int
    dtype: str = "f32"             # storage type of x and dy ("f32" | "bf16"); w is f32
    agp_mode: int = 0              # 0 Bernoulli (the paper), 1 top-k, 2 off
    seed: int = 0                  # data seed of layer 0; layer i uses seed + i
    philox_seed: int = 0
    notes: str = ""


def round_to_bf16(a):
    """float32 -> nearest bfloat16 value (ties to even), returned as float32."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32)


def draw_layer(layer, recipe, seed, dtype="f32"):
    """Draw (x, w, dy) float32 arrays for one layer; see the module docstring for the order."""
    rng = np.random.default_rng(seed)
    x = rng.standard_normal(layer.x_shape, dtype=np.float32)
    w = rng.standard_normal(layer.w_shape, dtype=np.float32)
    z = rng.standard_normal(layer.dy_shape, dtype=np.float32) if recipe.kind != "student_t" else None
    if recipe.kind == "sample_lognormal":
        s = np.exp(recipe.sigma * rng.standard_normal(layer.N)).astype(np.float32)
        if recipe.outlier_count:
            idx = rng.choice(layer.N, recipe.outlier_count, replace=False)
            s[idx] *= np.float32(recipe.outlier_factor)
        dy = z * s.reshape((layer.N,) + (1,) * (z.ndim - 1))
    elif recipe.kind == "channel_lognormal":
        s = np.exp(recipe.sigma * rng.standard_normal(layer.D)).astype(np.float32)
        dy = z * s.reshape((1, layer.D) + (1,) * (z.ndim - 2))
    elif recipe.kind == "student_t":
        dy = rng.standard_t(recipe.df, layer.dy_shape).astype(np.float32)
    elif recipe.kind == "sample_geometric":
        s = np.power(np.float64(recipe.ratio), np.arange(layer.N)).astype(np.float32)
        dy = z * s.reshape((layer.N,) + (1,) * (z.ndim - 1))
    else:
        raise ValueError(recipe.kind)
    dy = dy.astype(np.float32)
    if dtype == "bf16":
        x, dy = round_to_bf16(x), round_to_bf16(dy)
    return x, w, dy


# ----------------------------------------------------------------------------- layer lists

def resnet18_imagenet_arch(N=128, res=32, classes=10):
    """ResNet-18 with the ImageNet stem (7x7/2 conv, 3x3/2 max-pool) at input res x res:
    20 convolutions (incl. the three 1x1/2 shortcut projections) and the final fc."""
    L = []
    h = (res + 2 * 3 - 7) // 2 + 1
    L.append(LayerShape("conv1", "conv2d", N, 3, 64, res, res, 7, 7, 2, 2, 3, 3))
    h = (h + 2 * 1 - 3) // 2 + 1                      # max-pool 3x3/2 pad 1
    c = 64
    for stage, d in enumerate((64, 128, 256, 512), start=1):
        for blk in range(2):
            s = 2 if (stage > 1 and blk == 0) else 1
            ho = (h + 2 - 3) // s + 1
            L.append(LayerShape(f"l{stage}.{blk}.c1", "conv2d", N, c, d, h, h, 3, 3, s, s, 1, 1))
            L.append(LayerShape(f"l{stage}.{blk}.c2", "conv2d", N, d, d, ho, ho, 3, 3, 1, 1, 1, 1))
            if s != 1 or c != d:
                L.append(LayerShape(f"l{stage}.{blk}.down", "conv2d", N, c, d, h, h, 1, 1, s, s, 0, 0))
            c, h = d, ho
    L.append(LayerShape("fc", "linear", N, 512, classes))
    return tuple(L)


def vgg16_224(N=64, classes=1000):
    """VGG-16 at 224x224: 13 3x3/1 pad-1 convolutions and fc6 (25088->4096), fc7, fc8."""
    cfg = [(3, 64, 224), (64, 64, 224), (64, 128, 112), (128, 128, 112), (128, 256, 56),
           (256, 256, 56), (256, 256, 56), (256, 512, 28), (512, 512, 28), (512, 512, 28),
           (512, 512, 14), (512, 512, 14), (512, 512, 14)]
    L = [LayerShape(f"conv{i + 1}", "conv2d", N, c, d, h, h, 3, 3, 1, 1, 1, 1)
         for i, (c, d, h) in enumerate(cfg)]
    L += [LayerShape("fc6", "linear", N, 25088, 4096), LayerShape("fc7", "linear", N, 4096, 4096),
          LayerShape("fc8", "linear", N, 4096, classes)]
    return tuple(L)


WORKLOADS = {
    "linear_32x256x128": Workload(
        "linear_32x256x128",
        (LayerShape("fc", "linear", 32, 256, 128),),
        Recipe("sample_lognormal", sigma=1.5), bits=2,
        notes="single linear layer, per-sample lognormal(0,1.5) gradient scale, keep 1/2"),
    "vgg_cifar_conv3x3_256": Workload(
        "vgg_cifar_conv3x3_256",
        (LayerShape("conv", "conv2d", 128, 256, 256, 8, 8, 3, 3, 1, 1, 1, 1),),
        Recipe("sample_lognormal", sigma=2.0, outlier_count=13, outlier_factor=100.0), bits=4,
        notes="VGG-16 CIFAR-shaped 3x3 conv 256->256 on 8x8, N=128; per-sample lognormal(0,2) "
              "scale, 13 of 128 samples x100; keep 1/4"),
    "resnet18_32px": Workload(
        "resnet18_32px", resnet18_imagenet_arch(), Recipe("student_t", df=3.0), bits=4,
        notes="ResNet-18 (ImageNet stem) at 32x32, N=128, Student-t(3) gradients; b=4"),
    "vgg16_224_bf16": Workload(
        "vgg16_224_bf16", vgg16_224(), Recipe("channel_lognormal", sigma=1.5), bits=2,
        dtype="bf16",
        notes="VGG-16 at 224x224, N=64, bf16 x/dy/dx, per-channel lognormal(0,1.5); keep 1/2"),
}


def gemm_sweep_points():
    """(M, N, K) points of the binary GEMM sweep (M = N)."""
    return [(m, m, k) for m in (1024, 4096, 8192, 16384) for k in (2304, 4608, 16384)]


def draw_bits(shape, seed):
    """Uniform random bits (Bernoulli 1/2) as a bool array."""
    return np.random.default_rng(seed).integers(0, 2, size=shape, dtype=np.uint8).astype(bool)
