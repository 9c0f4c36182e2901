"""Pins for the ResNet-50-shaped forward (config: batch 64, 224x224, G=8 K=2).

The paper gives no ResNet-50 numbers; the network description is pinned to
the published ResNet-50 counts, and the oracle's composition to torch's
float64 functional convolution / pooling on a reduced input."""
import numpy as np
import pytest
import torch

import oracle
import oracle.resnet as orn
from paper_1910_11971_amd import workloads as wl


def spatial_plan(layers, hw):
    """(input size, output size) of every conv, following the network order."""
    out = {}
    def o(h, L):
        return (h + 2 * L.pad - L.k) // L.stride + 1
    h1 = o(hw, layers[0])
    out[0] = (hw, h1)
    h = (h1 + 2 - 3) // 2 + 1
    i = 1
    while i < len(layers):
        ds = i + 3 < len(layers) and layers[i + 3].name.endswith(".ds")
        out[i] = (h, h)
        h2 = o(h, layers[i + 1])
        out[i + 1] = (h, h2)
        out[i + 2] = (h2, h2)
        if ds:
            out[i + 3] = (h, o(h, layers[i + 3]))
        h = h2
        i += 4 if ds else 3
    return out, h


def test_layer_table_matches_published_resnet50_counts():
    L = wl.resnet50_layers()
    assert len(L) == 53
    conv_w = sum(l.Cout * l.fan_in for l in L)
    assert conv_w == 23_454_912
    # + FC weight and bias + batch-norm gamma/beta: the usual 25.56 M total
    assert conv_w + 2048 * 1000 + 1000 + 2 * sum(l.Cout for l in L) == 25_557_032
    plan, final = spatial_plan(L, 224)
    assert final == 7
    macs = sum(plan[i][1] ** 2 * l.Cout * l.fan_in for i, l in enumerate(L))
    assert macs == 4_087_136_256            # conv MACs per image
    assert macs + 2048 * 1000 == 4_089_184_256


def test_cci_layers_keep_k_of_g():
    L = wl.resnet50_layers(8, 2)
    assert L[0].K == 8 and all(l.K == 2 for l in L[1:])
    assert sum(1 for l in L if l.name.endswith(".ds")) == 4
    assert all((l.residual != "") == l.name.endswith(".c3") for l in L)


def _torch_reference(X, layers, ws, fcw, G, scales, biases):
    """Same network with torch float64 ops (NCHW), bf16 rounding via torch."""
    def rnd(t):
        return t.to(torch.float32).to(torch.bfloat16).to(torch.float64)

    def conv(i, x, res=None):
        L = layers[i]
        Wm = orn.masked_weight(ws[i], G, L.K).reshape(L.Cout, L.k, L.k, L.Cin)
        Wt = torch.from_numpy(Wm.astype(np.float64)).permute(0, 3, 1, 2)
        y = torch.nn.functional.conv2d(x, Wt, stride=L.stride, padding=L.pad)
        y = y * torch.from_numpy(scales[i].astype(np.float64)).view(1, -1, 1, 1)
        y = y + torch.from_numpy(biases[i].astype(np.float64)).view(1, -1, 1, 1)
        if res is not None:
            y = y + res
        if L.relu:
            y = torch.relu(y)
        return rnd(y)

    x = torch.from_numpy(np.asarray(X, np.float64)).permute(0, 3, 1, 2)
    x = conv(0, x)
    x = torch.nn.functional.max_pool2d(x, 3, 2, 1)
    i = 1
    while i < len(layers):
        ds = i + 3 < len(layers) and layers[i + 3].name.endswith(".ds")
        y = conv(i + 1, conv(i, x))
        ident = conv(i + 3, x) if ds else x
        x = conv(i + 2, y, ident)
        i += 4 if ds else 3
    pooled = rnd(x.mean(dim=(2, 3)))
    Wfc = torch.from_numpy(orn.masked_weight(fcw, G, G).astype(np.float64))
    return (pooled @ Wfc.T).numpy()


def test_oracle_forward_matches_torch_float64_reduced_input():
    net = wl.ResNet50(B=1, HW=32)
    X, ws, fcw = wl.draw_resnet50(net)
    sc = [wl.bn_fold(l.Cout)[0] for l in net.layers]
    bi = [wl.bn_fold(l.Cout)[1] for l in net.layers]
    Xf = X.float().numpy()
    got = orn.resnet50_forward(Xf, net.layers, ws, fcw, net.G, sc, bi)
    ref = _torch_reference(Xf, net.layers, ws, fcw, net.G, sc, bi)
    assert got.shape == (1, 1000)
    err = np.abs(got - ref).max() / np.abs(ref).max()
    assert err < 1e-6, err


def test_masked_weight_keeps_k_per_group_and_drops_the_rest():
    rng = np.random.default_rng(3)
    W = rng.standard_normal((64, 72)).astype(np.float32)
    Wm = orn.masked_weight(W, 8, 2)
    nz = (Wm.reshape(8, 8, 72) != 0).sum(axis=1)
    assert (nz == 2).all()
    kept = Wm != 0
    assert np.array_equal(Wm[kept], orn.round_bf16(W)[kept])
