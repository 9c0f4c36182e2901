"""MobileNetV2 pointwise layers (CCI on 1x1 convs, G = 8, s = 1..4) on the
GPU vs the oracle: every distinct layer shape at a reduced image size, and
the largest layers at batch 64 (every output)."""
import numpy as np
import pytest
import torch

from gpu_common import need_gpu, rand_epilogue
from test_gpu_conv import run_conv
from paper_1910_11971_amd import workloads as wl

pytestmark = pytest.mark.gpu

SHAPES = sorted({(l.Cin, l.Cout, l.kind) for l in wl.mobilenetv2_cci_layers()})


@pytest.mark.parametrize("K", [1, 2, 3, 4])
@pytest.mark.parametrize("Cin,Cout,kind", SHAPES)
def test_pointwise_layer_shapes(Cin, Cout, kind, K):
    """3 images of 10x11 (330 pixels: several tiles and a ragged tail), the
    route the network takes (auto), batch norm folded into scale / bias;
    ReLU after expanding layers, a residual on projecting layers that keep
    the channel count."""
    need_gpu()
    w = wl.conv("t", 3, 10, 11, Cin, Cout, 1, 1, 0, G=8, K=K,
                x_dist="relu_normal" if kind == "project" else "normal",
                w_std=(2.0 / Cin) ** 0.5, seed=100 * K + Cin)
    X, W = wl.draw(w)
    ep = rand_epilogue(Cout, w.N, torch.bfloat16, 7 + K, residual=(kind == "project" and Cin == Cout),
                       relu=(kind == "expand"))
    run_conv(X, W, 8, K, 1, 1, 0, torch.bfloat16, "auto", ep=ep)


@pytest.mark.parametrize("K", [3, 1])
@pytest.mark.parametrize("name", ["b2.0.expand", "b2.0.project", "b2.1.expand", "b6.2.project",
                                  "b7.0.project"])
def test_pointwise_layer_batch64_every_output(name, K):
    """Batch-64 layers as the sweep runs them (the largest pixel counts,
    C = 16 / 96 / 24 / 960), every output."""
    need_gpu()
    P = {w.name: w for w in wl.mobilenetv2_pointwise(B=64, K=K)}
    w = P["mbv2." + name]
    X, W = wl.draw(w)
    run_conv(X, W, w.G, w.K, 1, 1, 0, torch.bfloat16, "auto")
