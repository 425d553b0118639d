"""Seeded synthetic inputs for pattern-sparse 3x3 convolution workloads.

This module only draws numbers and describes shapes: it holds none of the
method's arithmetic (no projection, selection, packing or convolution), so the
HIP path and the CPU oracle can both take their inputs from it.

Distributions follow the paper where it fixes them and the workload
definitions otherwise:
  * activations ~ N(0, 1), except the first layer of the VGG-16 stack, whose
    pixels are discrete-uniform integers 0..255 -- the synthetic images of
    Sec. 4.1 and Sec. 5.1 of Gong et al. (GLSVLSI'20);
  * weights ~ N(0, sqrt(2 / (9 * Cin))) (He initialisation);
  * optional bias ~ N(0, 0.1);
  * fp16 data is drawn in fp32 and rounded to nearest-even binary16.

Seeds are ``1000 * workload.seed_base + 10 * layer + {0: W, 1: x, 2: bias}``
with numpy's PCG64, so every array is reproducible by name.
"""
from __future__ import annotations

import dataclasses
from typing import List, Optional, Sequence, Tuple

import numpy as np

DTYPES = {"f32": np.float32, "f16": np.float16}


@dataclasses.dataclass(frozen=True)
class ConvLayer:
    """One 3x3, pad-1 layer of a workload (h, w: input size)."""
    name: str
    cin: int
    cout: int
    h: int
    w: int
    keep: int            # beta: exact number of kernels kept
    relu: bool = False
    pool_after: bool = False   # 2x2/2 max-pool follows (VGG stack only)
    stride: int = 1            # 2: output (h-1)//2+1 x (w-1)//2+1 (ResNet stage entries)

    @property
    def out_hw(self) -> Tuple[int, int]:
        return (self.h - 1) // self.stride + 1, (self.w - 1) // self.stride + 1

    @property
    def n_kernels(self) -> int:
        return self.cin * self.cout


@dataclasses.dataclass(frozen=True)
class Workload:
    """A named stack of layers run at one batch size and one dtype."""
    name: str
    seed_base: int
    batch: int
    dtype: str                     # "f32" or "f16"
    m: int                         # pattern-library size
    layers: Tuple[ConvLayer, ...]
    x_dist: str = "normal"         # "normal" or "pixels" (first layer only)
    chained: bool = False          # layer l+1 consumes layer l's output

    @property
    def np_dtype(self):
        return DTYPES[self.dtype]


def keep_after_drop(n_kernels: int, drop_percent: int) -> int:
    """Kernels kept when ``drop_percent`` % are removed (exact integers)."""
    dropped = (n_kernels * drop_percent + 99) // 100
    return n_kernels - dropped


def keep_fraction(n_kernels: int, num: int, den: int) -> int:
    """floor(n_kernels * num / den), exact."""
    return (n_kernels * num) // den


# ---------------------------------------------------------------- workloads
def single_layer_64() -> Workload:
    """One 64->64 layer on a 1x64x32x32 fp32 input, 8 patterns, 50 % of the
    kernels dropped."""
    k = 64 * 64
    return Workload("single_64c_32x32_b1_f32", 1, 1, "f32", 8,
                    (ConvLayer("conv", 64, 64, 32, 32, keep_after_drop(k, 50)),))


def vgg16_stack(batch: int = 1) -> Workload:
    """The 13 3x3 layers of VGG-16 on a 224x224 image, fp32, ReLU after each
    layer, 2x2 max-pool after layers 2, 4, 7 and 10; the first layer keeps
    all its kernels, every later one keeps floor(K / 3)."""
    spec = [(3, 64, 224), (64, 64, 224), (64, 128, 112), (128, 128, 112),
            (128, 256, 56), (256, 256, 56), (256, 256, 56),
            (256, 512, 28), (512, 512, 28), (512, 512, 28),
            (512, 512, 14), (512, 512, 14), (512, 512, 14)]
    pools = {1, 3, 6, 9}
    layers = []
    for i, (cin, cout, s) in enumerate(spec):
        k = cin * cout
        keep = k if i == 0 else keep_fraction(k, 1, 3)
        layers.append(ConvLayer("conv%d" % (i + 1), cin, cout, s, s, keep,
                                relu=True, pool_after=i in pools))
    return Workload("vgg16_224_b%d_f32" % batch, 2, batch, "f32", 8,
                    tuple(layers), x_dist="pixels", chained=True)


def resnet50_3x3(batch: int) -> Workload:
    """The 16 3x3 convolutions of ResNet-50's bottlenecks, all at stride 1
    with Cin = Cout: 3 x 64@56, 4 x 128@28, 6 x 256@14, 3 x 512@7; fp16
    storage, 8 patterns, 60 % of kernels dropped."""
    layers = []
    for c, s, cnt in ((64, 56, 3), (128, 28, 4), (256, 14, 6), (512, 7, 3)):
        for j in range(cnt):
            layers.append(ConvLayer("c%d_s%d_%d" % (c, s, j), c, c, s, s,
                                    keep_after_drop(c * c, 60)))
    return Workload("resnet50_3x3_b%d_f16" % batch, 3, batch, "f16", 8, tuple(layers))


def resnet18_cifar_3x3(batch: int = 256) -> Workload:
    """The 16 3x3 convolutions of a CIFAR-shaped ResNet-18 (4 each of 64@32,
    128@16, 256@8, 512@4), fp32, 6 patterns, 70 % of kernels dropped."""
    layers = []
    for c, s in ((64, 32), (128, 16), (256, 8), (512, 4)):
        for j in range(4):
            layers.append(ConvLayer("c%d_s%d_%d" % (c, s, j), c, c, s, s,
                                    keep_after_drop(c * c, 70)))
    return Workload("resnet18_cifar_3x3_b%d_f32" % batch, 4, batch, "f32", 6, tuple(layers))


def resnet18_cifar_entry(batch: int = 256) -> Workload:
    """The 3x3 convolutions of a CIFAR-shaped ResNet-18 that change the
    channel count: the stem 3->64 at 32x32 (stride 1, every kernel kept) and
    the stride-2 stage entries 64->128 at 32x32, 128->256 at 16x16 and
    256->512 at 8x8 (70 % of kernels dropped); fp32, 6 patterns."""
    layers = [ConvLayer("stem", 3, 64, 32, 32, 3 * 64, relu=True)]
    for ci, s in ((64, 32), (128, 16), (256, 8)):
        layers.append(ConvLayer("entry%d_s%d" % (2 * ci, s), ci, 2 * ci, s, s,
                                keep_after_drop(ci * 2 * ci, 70), relu=True, stride=2))
    return Workload("resnet18_cifar_entry_b%d_f32" % batch, 6, batch, "f32", 6, tuple(layers))


def sweep_512(m: int, drop: int, batch: int = 64) -> Workload:
    """One 512->512 layer at 28x28, fp16, library size m, drop ratio drop %."""
    return Workload("sweep_512c_28x28_b%d_f16_m%d_d%d" % (batch, m, drop), 5, batch,
                    "f16", m,
                    (ConvLayer("conv", 512, 512, 28, 28,
                               keep_after_drop(512 * 512, drop)),))


def all_workloads() -> List[Workload]:
    out = [single_layer_64(), vgg16_stack(1), resnet50_3x3(1), resnet50_3x3(32),
           resnet18_cifar_3x3(256), resnet18_cifar_entry(256)]
    for m in (4, 8, 12):
        for d in (0, 40, 60, 80):
            out.append(sweep_512(m, d))
    return out


# ---------------------------------------------------------------- drawing
def _rng(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed))


def seed_of(wl: Workload, layer: int, what: str) -> int:
    return 1000 * wl.seed_base + 10 * layer + {"w": 0, "x": 1, "bias": 2}[what]


def he_weights(seed: int, cout: int, cin: int, dtype=np.float32) -> np.ndarray:
    """OIHW [cout][cin][3][3] weights ~ N(0, sqrt(2 / (9 cin)))."""
    std = np.float32(np.sqrt(2.0 / (9.0 * cin)))
    w = _rng(seed).standard_normal((cout, cin, 3, 3), dtype=np.float32) * std
    return w.astype(dtype)


def normal_activations(seed: int, shape: Sequence[int], dtype=np.float32) -> np.ndarray:
    return _rng(seed).standard_normal(tuple(shape), dtype=np.float32).astype(dtype)


def pixel_activations(seed: int, shape: Sequence[int], dtype=np.float32) -> np.ndarray:
    """Discrete-uniform integers 0..255 inclusive, stored as floats."""
    return _rng(seed).integers(0, 256, size=tuple(shape)).astype(dtype)


def bias_vector(seed: int, cout: int, dtype=np.float32) -> np.ndarray:
    return (_rng(seed).standard_normal(cout, dtype=np.float32)
            * np.float32(0.1)).astype(dtype)


def layer_weights(wl: Workload, li: int) -> np.ndarray:
    lay = wl.layers[li]
    return he_weights(seed_of(wl, li, "w"), lay.cout, lay.cin, wl.np_dtype)


def layer_input(wl: Workload, li: int, batch: Optional[int] = None) -> np.ndarray:
    """Input of layer ``li`` drawn on its own (for per-layer runs of a chained
    stack the later layers get non-negative N(0,1) magnitudes, the value range
    a ReLU output has)."""
    lay = wl.layers[li]
    n = wl.batch if batch is None else batch
    shape = (n, lay.cin, lay.h, lay.w)
    seed = seed_of(wl, li, "x")
    if wl.x_dist == "pixels" and li == 0:
        return pixel_activations(seed, shape, wl.np_dtype)
    x = normal_activations(seed, shape, wl.np_dtype)
    if wl.chained and li > 0:
        x = np.abs(x)
    return x


def layer_bias(wl: Workload, li: int) -> np.ndarray:
    return bias_vector(seed_of(wl, li, "bias"), wl.layers[li].cout, wl.np_dtype)


def all_kernels(wl: Workload) -> np.ndarray:
    """Every 3x3 kernel of the workload, concatenated as [K_total][3][3]
    (the scope the pattern library is chosen over)."""
    return np.concatenate([layer_weights(wl, i).reshape(-1, 3, 3)
                           for i in range(len(wl.layers))], axis=0)


def random_masks(seed: int, m: int, centre: bool = True) -> np.ndarray:
    """m distinct 4-of-9 masks (bit 3r+s), optionally all containing the
    centre, for tests that need a library not chosen from weights."""
    rng = _rng(seed)
    codes = [c for c in range(512) if bin(c).count("1") == 4 and (not centre or (c >> 4) & 1)]
    idx = rng.choice(len(codes), size=m, replace=False)
    return np.array([codes[i] for i in idx], dtype=np.uint16)


# ---------------------------------------------------------------- ADMM pruning
@dataclasses.dataclass(frozen=True)
class AdmmWorkload:
    """One layer pruned by data-free ADMM (Algorithm 1) on batches of T
    synthetic inputs: the layer's pre-trained weights and bias are He-init
    and N(0, 0.1) draws; each iteration k draws a new batch."""
    name: str
    seed_base: int
    batch: int                 # T
    layer: ConvLayer
    m: int
    x_dist: str                # "pixels": U{0..255} / 255; "relu": |N(0, 1)|
    lr: float = 1e-3

    def weights(self) -> np.ndarray:
        return he_weights(1000 * self.seed_base, self.layer.cout, self.layer.cin)

    def bias(self) -> np.ndarray:
        return bias_vector(1000 * self.seed_base + 2, self.layer.cout)

    def batch_input(self, k: int) -> np.ndarray:
        """Batch of iteration k (from 1): images with U{0..255} pixels scaled
        to [0, 1] for a first layer, or non-negative N(0,1) magnitudes (the
        value range of a ReLU output) for a later one."""
        shape = (self.batch, self.layer.cin, self.layer.h, self.layer.w)
        seed = 1000 * self.seed_base + 100 + k
        if self.x_dist == "pixels":
            return (pixel_activations(seed, shape) / np.float32(255.0)).astype(np.float32)
        return np.abs(normal_activations(seed, shape))


def admm_workloads() -> List[AdmmWorkload]:
    """VGG-16's first layer (3->64 at 224x224, every kernel kept: pattern
    pruning only) on synthetic images, and a 64->64 layer at 32x32 with half
    of its kernels dropped (patterns + connectivity), both at T = 32."""
    return [
        AdmmWorkload("admm_vgg16_conv1_T32", 7, 32, ConvLayer("conv1", 3, 64, 224, 224, 3 * 64, relu=True), 8,
                     "pixels"),
        AdmmWorkload("admm_64c_32x32_T32", 8, 32,
                     ConvLayer("conv", 64, 64, 32, 32, keep_after_drop(64 * 64, 50), relu=True), 8, "relu"),
    ]
