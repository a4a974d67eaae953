"""Seeded synthetic inputs and workload shapes.

This module is shared by the GPU path's tests and benchmark *and* by the
oracle's tests, so it holds no convolution arithmetic at all: only random
draws, storage-format quantisation of those draws (the bits handed to both
sides), decoding of half-precision bits, and the table of layer shapes.

Workloads stand in for the paper's ImageNet / ResNet-50 training runs
(Sec. 4, Table 1): no dataset is read; activations, weights and gradients are
drawn from the distributions below with the shapes of ResNet-50 v1.5's 53
convolution layers.
"""
from __future__ import annotations

import dataclasses
import math
from typing import List, Tuple

import numpy as np

F16 = "f16"
BF16 = "bf16"


# ---------------------------------------------------------------------------
# draws and storage formats
# ---------------------------------------------------------------------------

def generator(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(int(seed)))


def seed_for(cfg: int, layer: int, which: str) -> int:
    """Seed = 1_000_000*config + 1000*layer + {x:1, w:2, dy:3, old:4}."""
    return 1_000_000 * int(cfg) + 1000 * int(layer) + {"x": 1, "w": 2, "dy": 3, "old": 4}[which]


def to_bits(v: np.ndarray, dtype: str) -> np.ndarray:
    """Round-to-nearest-even quantisation of float values to fp16 or bf16,
    returned as raw uint16 bit patterns."""
    if dtype == F16:
        with np.errstate(over="ignore"):  # values past the fp16 range round to +-inf
            return np.asarray(v).astype(np.float16).view(np.uint16)
    if dtype == BF16:
        f = np.ascontiguousarray(v, dtype=np.float32)
        b = f.view(np.uint32).astype(np.uint64)
        nan = np.isnan(f)
        rounded = (b + 0x7FFF + ((b >> 16) & 1)) >> 16
        out = rounded.astype(np.uint16)
        out[nan] = 0x7FC0
        return out
    raise ValueError("dtype must be 'f16' or 'bf16'")


def from_bits(bits: np.ndarray, dtype: str) -> np.ndarray:
    """Exact float64 values of fp16 / bf16 bit patterns."""
    bits = np.ascontiguousarray(bits, dtype=np.uint16)
    if dtype == F16:
        return bits.view(np.float16).astype(np.float64)
    if dtype == BF16:
        with np.errstate(invalid="ignore"):
            return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    raise ValueError("dtype must be 'f16' or 'bf16'")


def draw(seed: int, shape, kind: str, scale: float = 1.0, dtype: str = F16) -> np.ndarray:
    """Seeded draw quantised to ``dtype``; returns uint16 bits.

    kind: 'normal'  -> scale * N(0, 1)
          'absnormal' -> scale * |N(0, 1)|   (ReLU-like activations)
    """
    g = generator(seed)
    v = g.standard_normal(size=shape, dtype=np.float32)
    if kind == "absnormal":
        np.abs(v, out=v)
    elif kind != "normal":
        raise ValueError(kind)
    if scale != 1.0:
        v *= np.float32(scale)
    return to_bits(v, dtype)


def he_std(fan_in: int) -> float:
    """He-normal standard deviation sqrt(2 / fan_in)."""
    return math.sqrt(2.0 / fan_in)


# ---------------------------------------------------------------------------
# shapes
# ---------------------------------------------------------------------------

@dataclasses.dataclass(frozen=True)
class Layer:
    name: str
    n: int
    c: int
    h: int
    w: int
    k: int
    r: int
    s: int
    stride: int = 1
    pad: int = 0
    dil: int = 1
    groups: int = 1
    c_logical: int = 0      # channel count before padding (stem: 3 padded to 4)
    count: int = 1          # how many ResNet-50 layers share this shape
    dgrad: bool = True      # the stem has no gradient to the image
    # width-axis stride / padding / dilation when they differ from the
    # height axis (0, -1, 0: the same as stride, pad, dil)
    stride_w: int = 0
    pad_w: int = -1
    dil_w: int = 0

    @property
    def s_w(self) -> int:
        return self.stride_w or self.stride

    @property
    def p_w(self) -> int:
        return self.pad if self.pad_w < 0 else self.pad_w

    @property
    def d_w(self) -> int:
        return self.dil_w or self.dil

    @property
    def p(self) -> int:
        return (self.h + 2 * self.pad - self.dil * (self.r - 1) - 1) // self.stride + 1

    @property
    def q(self) -> int:
        return (self.w + 2 * self.p_w - self.d_w * (self.s - 1) - 1) // self.s_w + 1

    @property
    def c_alg(self) -> int:
        return self.c_logical or self.c

    def flops(self, executed: bool = False) -> int:
        """2*N*K*P*Q*(C/g)*R*S for one pass; the algorithmic count uses the
        logical channel count, the executed count the padded one."""
        c = self.c if executed else self.c_alg
        return 2 * self.n * self.k * self.p * self.q * (c // self.groups) * self.r * self.s

    def with_batch(self, n: int) -> "Layer":
        return dataclasses.replace(self, n=n)


def resnet50_layers(batch: int) -> List[Tuple[Layer, int]]:
    """ResNet-50 v1.5 (stride on the 3x3 conv of each down-sampling block):
    the 23 distinct convolution shapes with their multiplicities (sum 53).
    The stem's 3 input channels are padded to 4."""
    L = []
    def add(name, c, h, k, r, stride, pad, count, **kw):
        L.append(Layer(name, batch, c, h, h, k, r, r, stride, pad, count=count, **kw))
    add("stem", 4, 224, 64, 7, 2, 3, 1, c_logical=3, dgrad=False)
    add("s2b0a", 64, 56, 64, 1, 1, 0, 1)
    add("s2b0b", 64, 56, 64, 3, 1, 1, 3)
    add("s2b0c", 64, 56, 256, 1, 1, 0, 4)
    add("s2b1a", 256, 56, 64, 1, 1, 0, 2)
    add("s3b0a", 256, 56, 128, 1, 1, 0, 1)
    add("s3b0b", 128, 56, 128, 3, 2, 1, 1)
    add("s3b0c", 128, 28, 512, 1, 1, 0, 4)
    add("s3b0proj", 256, 56, 512, 1, 2, 0, 1)
    add("s3b1a", 512, 28, 128, 1, 1, 0, 3)
    add("s3b1b", 128, 28, 128, 3, 1, 1, 3)
    add("s4b0a", 512, 28, 256, 1, 1, 0, 1)
    add("s4b0b", 256, 28, 256, 3, 2, 1, 1)
    add("s4b0c", 256, 14, 1024, 1, 1, 0, 6)
    add("s4b0proj", 512, 28, 1024, 1, 2, 0, 1)
    add("s4b1a", 1024, 14, 256, 1, 1, 0, 5)
    add("s4b1b", 256, 14, 256, 3, 1, 1, 5)
    add("s5b0a", 1024, 14, 512, 1, 1, 0, 1)
    add("s5b0b", 512, 14, 512, 3, 2, 1, 1)
    add("s5b0c", 512, 7, 2048, 1, 1, 0, 3)
    add("s5b0proj", 1024, 14, 2048, 1, 2, 0, 1)
    add("s5b1a", 2048, 7, 512, 1, 1, 0, 2)
    add("s5b1b", 512, 7, 512, 3, 1, 1, 2)
    return [(l, l.count) for l in L]


def efficientnet_b0_depthwise(batch: int) -> List[Tuple[Layer, int]]:
    """The 16 depthwise convolutions of EfficientNet-B0 (224x224 input): the
    MBConv blocks' k x k depthwise stage, one group per channel, with the
    expanded channel counts, the stride on each stage's first block and
    "same" padding k // 2.  Distinct shapes with their multiplicities."""
    L = []
    def add(name, c, h, k, stride, count):
        L.append(Layer(name, batch, c, h, h, c, k, k, stride, k // 2, groups=c, count=count))
    add("mb1_dw3", 32, 112, 3, 1, 1)
    add("mb2a_dw3", 96, 112, 3, 2, 1)
    add("mb2b_dw3", 144, 56, 3, 1, 1)
    add("mb3a_dw5", 144, 56, 5, 2, 1)
    add("mb3b_dw5", 240, 28, 5, 1, 1)
    add("mb4a_dw3", 240, 28, 3, 2, 1)
    add("mb4b_dw3", 480, 14, 3, 1, 2)
    add("mb5a_dw5", 480, 14, 5, 1, 1)
    add("mb5b_dw5", 672, 14, 5, 1, 2)
    add("mb6a_dw5", 672, 14, 5, 2, 1)
    add("mb6b_dw5", 1152, 7, 5, 1, 3)
    add("mb7_dw3", 1152, 7, 3, 1, 1)
    return [(l, l.count) for l in L]


def resnext50_grouped(batch: int) -> List[Tuple[Layer, int]]:
    """The 16 grouped 3x3 convolutions of ResNeXt-50 (32x4d) at 224x224: 32
    groups of 4, 8, 16 and 32 channels in the four stages, the stride on the
    3x3 of each down-sampling block (as in ResNet-50 v1.5).  Distinct shapes
    with their multiplicities."""
    L = []
    def add(name, c, h, stride, count):
        L.append(Layer(name, batch, c, h, h, c, 3, 3, stride, 1, groups=32, count=count))
    add("x2_g4", 128, 56, 1, 3)
    add("x3a_g8", 256, 56, 2, 1)
    add("x3b_g8", 256, 28, 1, 3)
    add("x4a_g16", 512, 28, 2, 1)
    add("x4b_g16", 512, 14, 1, 5)
    add("x5a_g32", 1024, 14, 2, 1)
    add("x5b_g32", 1024, 7, 1, 2)
    return [(l, l.count) for l in L]


# The workloads: shapes, layout, dtype, distributions, loss scale.
@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    layers: Tuple[Layer, ...]
    layout: str            # "nchw" or "nhwc"
    dtype: str             # operand dtype
    loss_scale: float
    x_kind: str            # 'normal' | 'absnormal'
    x_scale: float
    w_scale: str           # 'he' or a float given as string
    dy_std: float          # dy = loss_scale * N(0, dy_std)  (scaled before quantisation)
    passes: Tuple[str, ...] = ("fwd", "dgrad", "wgrad")


def workload(cfg: int, dtype: str = F16, batch: int | None = None) -> Workload:
    """Config 1: tiny 3x3 NCHW; 2: ResNet-50 stage-1 bottleneck at batch 64;
    3: stage transitions at batch 128; 4: stem at batch 128; 5: all 53 layers
    at batch 256; 6: the depthwise layers of EfficientNet-B0 at batch 128
    (grouped convolution with one channel per group); 7: the grouped 3x3
    layers of ResNeXt-50 32x4d at batch 128."""
    if cfg == 1:
        n = batch or 2
        s = 1.0 / math.sqrt(16 * 9)
        return Workload("3x3 16->16 16x16 batch %d NCHW" % n,
                        (Layer("tiny3x3", n, 16, 16, 16, 16, 3, 3, 1, 1),),
                        "nchw", dtype, 1.0, "normal", s, repr(s), s)
    if cfg == 2:
        n = batch or 64
        ls = (Layer("1x1 256->64", n, 256, 56, 56, 64, 1, 1),
              Layer("3x3 64->64", n, 64, 56, 56, 64, 3, 3, 1, 1),
              Layer("1x1 64->256", n, 64, 56, 56, 256, 1, 1))
        return Workload("ResNet-50 stage-1 bottleneck batch %d" % n, ls, "nhwc", dtype,
                        1024.0, "absnormal", 1.0, "he", 1e-3)
    if cfg == 3:
        n = batch or 128
        ls = (Layer("3x3 128->128 s2", n, 128, 56, 56, 128, 3, 3, 2, 1),
              Layer("1x1 256->512 s2", n, 256, 56, 56, 512, 1, 1, 2, 0))
        return Workload("ResNet-50 stage transitions batch %d" % n, ls, "nhwc", dtype,
                        1024.0, "absnormal", 1.0, "he", 1e-3)
    if cfg == 4:
        n = batch or 128
        ls = (Layer("stem 7x7 3(4)->64 s2", n, 4, 224, 224, 64, 7, 7, 2, 3, c_logical=3,
                    dgrad=False),)
        return Workload("ResNet-50 stem batch %d" % n, ls, "nhwc", dtype, 1024.0,
                        "normal", 1.0, "he", 1e-3, passes=("fwd", "wgrad"))
    if cfg == 5:
        n = batch or 256
        ls = tuple(l for l, _ in resnet50_layers(n))
        return Workload("ResNet-50 all 53 conv layers batch %d" % n, ls, "nhwc", dtype,
                        1024.0, "absnormal", 1.0, "he", 1e-3)
    if cfg == 6:
        n = batch or 128
        ls = tuple(l for l, _ in efficientnet_b0_depthwise(n))
        return Workload("EfficientNet-B0 16 depthwise layers batch %d" % n, ls, "nhwc", dtype,
                        1024.0, "absnormal", 1.0, "he", 1e-3)
    if cfg == 7:
        n = batch or 128
        ls = tuple(l for l, _ in resnext50_grouped(n))
        return Workload("ResNeXt-50 32x4d 16 grouped 3x3 layers batch %d" % n, ls, "nhwc", dtype,
                        1024.0, "absnormal", 1.0, "he", 1e-3)
    raise ValueError("config must be 1..7")


def layer_tensors(wl: Workload, li: int, cfg: int, layer: Layer | None = None):
    """Seeded operands of one layer as uint16 bits in the workload's layout.

    Returns dict(x=..., w=..., dy=...).  x: [N,C,H,W] or [N,H,W,C]; w: [K,C/g,R,S]
    or [K,R,S,C/g]; dy: [N,K,P,Q] or [N,P,Q,K].  For a padded stem the pad
    channels of x and w are zero.  dy is drawn as loss_scale * N(0, dy_std)
    and quantised once; the loss scale is therefore already inside dy."""
    L = layer or wl.layers[li]
    cg = L.c // L.groups
    nchw = wl.layout == "nchw"
    cl = L.c_alg
    if nchw:
        xs, ws, dys = (L.n, cl, L.h, L.w), (L.k, cl // L.groups, L.r, L.s), (L.n, L.k, L.p, L.q)
    else:
        xs, ws, dys = (L.n, L.h, L.w, cl), (L.k, L.r, L.s, cl // L.groups), (L.n, L.p, L.q, L.k)
    x = draw(seed_for(cfg, li, "x"), xs, wl.x_kind, wl.x_scale, wl.dtype)
    wsd = he_std((cl // L.groups) * L.r * L.s) if wl.w_scale == "he" else float(wl.w_scale)
    w = draw(seed_for(cfg, li, "w"), ws, "normal", wsd, wl.dtype)
    dy = draw(seed_for(cfg, li, "dy"), dys, "normal", wl.loss_scale * wl.dy_std, wl.dtype)
    if cl != L.c:  # zero-pad channels (channel-last only)
        assert not nchw
        xp = np.zeros((L.n, L.h, L.w, L.c), np.uint16)
        xp[..., :cl] = x
        wp = np.zeros((L.k, L.r, L.s, cg), np.uint16)
        wp[..., :cl] = w
        x, w = xp, wp
    return dict(x=x, w=w, dy=dy)
