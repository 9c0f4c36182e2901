"""Seeded synthetic workloads shaped like the paper's CNN layers.

This module only draws random inputs; it holds none of the CCI method's
arithmetic and is the one piece shared by the HIP path's tests/benchmark and
the CPU oracle's checks.  Every draw uses numpy's PCG64 generator seeded per
workload, standard normal samples in float64, scaled, then rounded to fp32
(numpy cast, round-to-nearest-even) and, for bf16 inputs, rounded once more to
bfloat16 by torch's conversion.  Draw order: activations X first, then the
dense fp32 master weights W.

The layer shapes stand in for the paper's ImageNet / CIFAR CNN layers
(Sec. 6): no dataset is read.
  fc256      single FC layer, fp32, X [64,256] ~ N(0,1), W [256,256] ~ N(0,1/256),
             G=8, K=4 (50% sparse)
  conv3x3    3x3 conv, batch 32, 56x56, 64->64, pad 1, stride 1, X bf16 ~ N(0,1),
             W ~ N(0, 2/576), G=8, K=2 (75%), bf16 out (ResNet layer1 3x3)
  conv1x1    1x1 bottleneck conv, batch 64, 14x14, 1024->256, X bf16 ~ ReLU(N(0,1)),
             W ~ N(0, 2/1024), G=16, K=4 or 2 (75% / 87.5%)
  fc4096     FC sweep, X bf16 [4096,4096] ~ N(0,1), W [4096,4096] ~ N(0,1/4096),
             G=16, K in {1,2,4,8,16} (K=16 is the dense control)
  resnet50   ResNet-50-shaped forward (torchvision v1.5 layout: stride on the 3x3
             conv), images bf16 [B,224,224,3] ~ N(0,1); every conv He-initialised
             W ~ N(0, 2/fan_in) with CCI G=8, K=2 except the first conv (dense:
             K=G); batch norm at its initial state folded into the epilogue
             (scale 1/sqrt(1+1e-5), bias 0); FC 2048->1000 W ~ N(0, 1/2048),
             dense (K=G), fp32 logits.  Draw order: images, then every conv in
             network order (stem, then per bottleneck c1, c2, c3, downsample),
             then the FC.
  mobilenetv2 (pointwise)  the 32 sparse 1x1 convs of MobileNetV2 (width 1,
             224x224) at batch 64, G=8, K in {1,2,3,4}, each an independent
             layer: X bf16 ~ N(0,1) for expanding layers, ~ ReLU(N(0,1)) for
             projecting ones; W ~ N(0, 2/Cin); layer i seeded with seed + i.
"""
from __future__ import annotations

from dataclasses import dataclass, replace

import numpy as np


@dataclass(frozen=True)
class Workload:
    name: str
    # activations: FC uses (N, C); conv uses NHWC (B, H, W, Cin) and a kernel
    B: int
    H: int
    W: int
    Cin: int
    O: int
    KH: int = 1
    KW: int = 1
    stride: int = 1
    pad: int = 0
    G: int = 8
    K: int = 2
    x_dtype: str = "bf16"      # "f32" | "bf16"
    y_dtype: str = "bf16"      # "f32" | "bf16"
    x_dist: str = "normal"     # "normal" | "relu_normal"
    w_std: float = 1.0
    seed: int = 0
    conv: bool = False

    # GEMM view ------------------------------------------------------------
    @property
    def Ho(self) -> int:
        return (self.H + 2 * self.pad - self.KH) // self.stride + 1 if self.conv else self.H

    @property
    def Wo(self) -> int:
        return (self.W + 2 * self.pad - self.KW) // self.stride + 1 if self.conv else self.W

    @property
    def N(self) -> int:
        """GEMM rows: samples (FC) or output pixels (conv)."""
        return self.B * self.Ho * self.Wo

    @property
    def C(self) -> int:
        """GEMM reduction length: inputs (FC) or KH*KW*Cin (conv)."""
        return self.KH * self.KW * self.Cin

    @property
    def nnz(self) -> int:
        return self.O * self.C * self.K // self.G

    @property
    def x_shape(self):
        return (self.B, self.H, self.W, self.Cin) if self.conv else (self.B * self.H * self.W, self.Cin)

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)


def fc(name, N, C, O, **kw) -> Workload:
    return Workload(name=name, B=N, H=1, W=1, Cin=C, O=O, conv=False, **kw)


def conv(name, B, H, W, Cin, O, k, stride, pad, **kw) -> Workload:
    return Workload(name=name, B=B, H=H, W=W, Cin=Cin, O=O, KH=k, KW=k,
                    stride=stride, pad=pad, conv=True, **kw)


WORKLOADS = {
    "fc256": fc("fc256", 64, 256, 256, G=8, K=4, x_dtype="f32", y_dtype="f32",
                w_std=(1 / 256) ** 0.5),
    "conv3x3": conv("conv3x3", 32, 56, 56, 64, 64, 3, 1, 1, G=8, K=2,
                    w_std=(2 / 576) ** 0.5),
    "conv1x1_k4": conv("conv1x1_k4", 64, 14, 14, 1024, 256, 1, 1, 0, G=16, K=4,
                       x_dist="relu_normal", w_std=(2 / 1024) ** 0.5),
    "conv1x1_k2": conv("conv1x1_k2", 64, 14, 14, 1024, 256, 1, 1, 0, G=16, K=2,
                       x_dist="relu_normal", w_std=(2 / 1024) ** 0.5),
}
for _k in (1, 2, 4, 8, 16):
    WORKLOADS[f"fc4096_k{_k}"] = fc(f"fc4096_k{_k}", 4096, 4096, 4096, G=16, K=_k,
                                    w_std=(1 / 4096) ** 0.5)


def draw(wl: Workload):
    """Return (X, W): X a torch CPU tensor in wl.x_dtype with wl.x_shape,
    W the dense fp32 master weights as numpy [O, C] (conv: [O, KH*KW*Cin] in
    (kh, kw, cin) order)."""
    import torch

    rng = np.random.Generator(np.random.PCG64(wl.seed))
    x = rng.standard_normal(wl.x_shape)
    if wl.x_dist == "relu_normal":
        x = np.maximum(x, 0.0)
    x32 = x.astype(np.float32)
    X = torch.from_numpy(x32)
    if wl.x_dtype == "bf16":
        X = X.to(torch.bfloat16)
    w = rng.standard_normal((wl.O, wl.C)) * wl.w_std
    W = np.ascontiguousarray(w.astype(np.float32))
    return X, W


def draw_epilogue(wl: Workload, *, scale=True, bias=True, residual=False, seed_offset=1000):
    """Optional fused-epilogue operands: per-output fp32 scale and bias and a
    residual shaped like Y (in wl.y_dtype).  Drawn from their own stream."""
    import torch

    rng = np.random.Generator(np.random.PCG64(wl.seed + seed_offset))
    out = {}
    if scale:
        out["scale"] = torch.from_numpy((0.5 + rng.random(wl.O)).astype(np.float32))
    if bias:
        out["bias"] = torch.from_numpy((0.1 * rng.standard_normal(wl.O)).astype(np.float32))
    if residual:
        r = torch.from_numpy(rng.standard_normal((wl.N, wl.O)).astype(np.float32))
        out["residual"] = r.to(torch.bfloat16) if wl.y_dtype == "bf16" else r
    return out


def small(wl: Workload, **kw) -> Workload:
    """A reduced copy of a workload (same G, K, dtypes, distributions)."""
    return wl.with_(**kw)


# ---------------------------------------------------------------------------
# ResNet-50-shaped forward


@dataclass(frozen=True)
class ConvLayer:
    name: str
    Cin: int
    Cout: int
    k: int
    stride: int
    pad: int
    K: int                 # kept weights per group (K == G: dense)
    relu: bool             # ReLU in the epilogue
    residual: str = ""     # c3 only: "identity" or "downsample"

    @property
    def fan_in(self) -> int:
        return self.k * self.k * self.Cin


BN_EPS = 1e-5
RESNET50_STAGES = ((64, 256, 3, 1), (128, 512, 4, 2), (256, 1024, 6, 2), (512, 2048, 3, 2))


def resnet50_layers(G: int = 8, K: int = 2) -> list[ConvLayer]:
    """The 53 convolutions of ResNet-50 (v1.5) in network order."""
    layers = [ConvLayer("conv1", 3, 64, 7, 2, 3, G, True)]
    cin = 64
    for si, (mid, out, blocks, stride) in enumerate(RESNET50_STAGES):
        for bi in range(blocks):
            s = stride if bi == 0 else 1
            pre = f"layer{si + 1}.{bi}"
            ds = bi == 0
            layers.append(ConvLayer(f"{pre}.c1", cin, mid, 1, 1, 0, K, True))
            layers.append(ConvLayer(f"{pre}.c2", mid, mid, 3, s, 1, K, True))
            layers.append(ConvLayer(f"{pre}.c3", mid, out, 1, 1, 0, K, True,
                                    "downsample" if ds else "identity"))
            if ds:
                layers.append(ConvLayer(f"{pre}.ds", cin, out, 1, s, 0, K, False))
            cin = out
    return layers


@dataclass(frozen=True)
class ResNet50:
    B: int = 64
    HW: int = 224
    G: int = 8
    K: int = 2
    classes: int = 1000
    seed: int = 0

    @property
    def layers(self) -> list[ConvLayer]:
        return resnet50_layers(self.G, self.K)


def draw_resnet50(net: ResNet50):
    """Return (X, conv_weights, fc_weight): X torch bf16 NHWC [B, HW, HW, 3];
    conv_weights a list of fp32 numpy [Cout, k*k*Cin] ((kh, kw, cin) order),
    one per layer of ``net.layers``; fc_weight fp32 numpy [classes, 2048]."""
    import torch

    rng = np.random.Generator(np.random.PCG64(net.seed))
    x = rng.standard_normal((net.B, net.HW, net.HW, 3)).astype(np.float32)
    X = torch.from_numpy(x).to(torch.bfloat16)
    ws = []
    for L in net.layers:
        w = rng.standard_normal((L.Cout, L.fan_in)) * (2.0 / L.fan_in) ** 0.5
        ws.append(np.ascontiguousarray(w.astype(np.float32)))
    fc_in = RESNET50_STAGES[-1][1]
    fcw = rng.standard_normal((net.classes, fc_in)) * (1.0 / fc_in) ** 0.5
    return X, ws, np.ascontiguousarray(fcw.astype(np.float32))


def bn_fold(C: int):
    """Batch norm at its initial state (gamma 1, beta 0, mean 0, var 1) folded
    into a per-channel scale and bias (fp32 numpy)."""
    scale = np.full(C, 1.0 / np.sqrt(1.0 + BN_EPS), np.float32)
    return scale, np.zeros(C, np.float32)


# ---------------------------------------------------------------------------
# MobileNetV2: the network the paper sparsifies on its pointwise layers only
# (Sec. 6, G = 8, s = 1..4)

# inverted-residual stages of MobileNetV2 (Sandler et al. 2018, Table 2):
# (expansion t, output channels c, blocks n, stride of the first block s)
MBV2_STAGES = ((1, 16, 1, 1), (6, 24, 2, 2), (6, 32, 3, 2), (6, 64, 4, 2),
               (6, 96, 3, 1), (6, 160, 3, 2), (6, 320, 1, 1))


def round_channels(v: float, d: int = 8) -> int:
    """Channel count for a width multiplier: the nearest multiple of d (at
    least d), raised by d when rounding lost more than 10%."""
    n = max(d, int(v + d / 2) // d * d)
    return n + d if n < 0.9 * v else n


@dataclass(frozen=True)
class NetLayer:
    name: str
    kind: str        # "stem" | "expand" | "depthwise" | "project" | "last" | "fc"
    Cin: int
    Cout: int
    k: int
    stride: int
    H: int           # input height (= width)
    residual: bool = False   # project layers: output added to the block input

    @property
    def Ho(self) -> int:
        if self.kind == "fc":
            return 1
        return (self.H + 2 * (self.k // 2) - self.k) // self.stride + 1

    @property
    def weights(self) -> int:
        """Weight (and, for the classifier, bias) parameters; batch norm not counted."""
        if self.kind == "depthwise":
            return self.k * self.k * self.Cout
        if self.kind == "fc":
            return self.Cin * self.Cout + self.Cout
        return self.k * self.k * self.Cin * self.Cout

    @property
    def macs(self) -> int:
        """Multiply-accumulates per image."""
        if self.kind == "fc":
            return self.Cin * self.Cout
        per_px = self.k * self.k * (self.Cout if self.kind == "depthwise" else self.Cin * self.Cout)
        return per_px * self.Ho * self.Ho


def mobilenetv2_layers(width: float = 1.0, res: int = 224, classes: int = 1000) -> list[NetLayer]:
    """Every weight layer of MobileNetV2 in network order: 3x3 stem (stride
    2), then per block an expanding 1x1 conv (absent when t = 1), a 3x3
    depthwise conv carrying the stride and a projecting 1x1 conv (residual
    when the stride is 1 and the channel count is kept), then a 1x1 conv to
    1280 channels, global pooling and the classifier."""
    L = [NetLayer("stem", "stem", 3, round_channels(32 * width), 3, 2, res)]
    h = L[0].Ho
    cin = L[0].Cout
    for si, (t, c, n, s) in enumerate(MBV2_STAGES):
        cout = round_channels(c * width)
        for bi in range(n):
            st = s if bi == 0 else 1
            hid = cin * t
            pre = f"b{si + 1}.{bi}"
            if t != 1:
                L.append(NetLayer(f"{pre}.expand", "expand", cin, hid, 1, 1, h))
            dw = NetLayer(f"{pre}.dw", "depthwise", hid, hid, 3, st, h)
            L.append(dw)
            h = dw.Ho
            L.append(NetLayer(f"{pre}.project", "project", hid, cout, 1, 1, h,
                              residual=(st == 1 and cin == cout)))
            cin = cout
    last = round_channels(1280 * max(1.0, width))
    L.append(NetLayer("last", "last", cin, last, 1, 1, h))
    L.append(NetLayer("fc", "fc", last, classes, 1, 1, 1))
    return L


def mobilenetv2_cci_layers(width: float = 1.0, res: int = 224) -> list[NetLayer]:
    """The pointwise layers that carry CCI sparsity: every expanding and
    projecting 1x1 conv of the inverted-residual blocks except the first
    block's projection (32 -> 16 at 112x112).  With that reading (and the
    1280-channel conv, the stem, the depthwise convs and the classifier
    dense) the network's weight and MAC counts agree with the paper's table
    of lightweight-architecture benchmarks (appendix) to 0.3%."""
    return [l for l in mobilenetv2_layers(width, res)
            if l.kind in ("expand", "project") and l.name != "b1.0.project"]


def mobilenetv2_pointwise(B: int = 64, K: int = 2, G: int = 8, res: int = 224, seed: int = 0) -> list[Workload]:
    """The CCI pointwise layers of MobileNetV2 at batch B as independent 1x1
    conv workloads (G, K from the paper's sweep).  Inputs of expanding layers
    are a projection's linear output ~ N(0,1); inputs of projecting layers
    follow a ReLU6 ~ ReLU(N(0,1)).  W ~ N(0, 2/Cin).  Layer i draws with seed
    + i."""
    out = []
    for i, l in enumerate(mobilenetv2_cci_layers(1.0, res)):
        out.append(conv(f"mbv2.{l.name}", B, l.H, l.H, l.Cin, l.Cout, 1, 1, 0, G=G, K=K,
                        x_dist="relu_normal" if l.kind == "project" else "normal",
                        w_std=(2.0 / l.Cin) ** 0.5, seed=seed + i))
    return out
