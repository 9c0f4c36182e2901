"""ResNet-50-shaped forward (config: batch 64, 224x224, CCI G=8 K=2, first conv
and classifier dense, folded batch norm, bf16 activations) against the
oracle: every layer on the GPU's own layer input at the full batch (every
output), and the logits end to end on a two-image batch (and on odd-sized
images)."""
import numpy as np
import pytest
import torch

import oracle
import oracle.resnet as orn
from gpu_common import DEV, epilogue_terms, need_gpu
from parity import TOL, check_close
from paper_1910_11971_amd import workloads as wl

pytestmark = pytest.mark.gpu


def _model(net):
    from paper_1910_11971_amd.resnet import ResNet50CCI
    X, ws, fcw = wl.draw_resnet50(net)
    return X, ws, fcw, ResNet50CCI(net, ws, fcw, device=DEV)


def _bn(net):
    return [wl.bn_fold(l.Cout)[0] for l in net.layers], [wl.bn_fold(l.Cout)[1] for l in net.layers]


def test_resnet50_logits_end_to_end_two_images():
    need_gpu()
    net = wl.ResNet50(B=2, HW=224)
    X, ws, fcw, model = _model(net)
    logits = model.forward(X.to(DEV))
    torch.cuda.synchronize()
    assert logits.dtype == torch.float32 and tuple(logits.shape) == (2, 1000)
    sc, bi = _bn(net)
    ref = orn.resnet50_forward(X.float().numpy(), net.layers, ws, fcw, net.G, sc, bi)
    got = logits.cpu().numpy()
    assert np.isfinite(got).all()
    rel = np.abs(got - ref).max() / np.abs(ref).max()
    assert rel <= TOL["bf16"], f"logits max|err|/max|ref| = {rel:.3e}"
    # the classifier's decision survives wherever the top-2 margin is clear
    top = np.argsort(-ref, axis=1)
    margin = ref[np.arange(2), top[:, 0]] - ref[np.arange(2), top[:, 1]]
    clear = margin > 4 * TOL["bf16"] * np.abs(ref).max()
    assert (got.argmax(1)[clear] == top[clear, 0]).all()


@pytest.mark.parametrize("HW", [37, 64])
def test_resnet50_logits_small_images(HW):
    """Odd and even input sizes: the first conv's zero-padded tap column must
    not change the output width (every layer's shape follows the 7x7 conv)."""
    need_gpu()
    net = wl.ResNet50(B=2, HW=HW)
    X, ws, fcw, model = _model(net)
    rec = []
    logits = model.forward(X.to(DEV), record=rec)
    torch.cuda.synchronize()
    Ho = (HW + 2 * 3 - 7) // 2 + 1
    assert tuple(rec[0][3].shape) == (2, Ho, Ho, 64)
    sc, bi = _bn(net)
    ref = orn.resnet50_forward(X.float().numpy(), net.layers, ws, fcw, net.G, sc, bi)
    got = logits.cpu().numpy()
    rel = np.abs(got - ref).max() / np.abs(ref).max()
    assert rel <= TOL["bf16"], f"HW={HW}: logits max|err|/max|ref| = {rel:.3e}"


def test_resnet50_every_layer_full_batch_every_output():
    """Each of the 53 convs on the GPU's own layer input at batch 64: every
    output pixel and channel against the oracle's direct convolution."""
    need_gpu()
    net = wl.ResNet50()  # batch 64, 224x224
    X, ws, fcw, model = _model(net)
    rec = []
    logits = model.forward(X.to(DEV), record=rec)
    torch.cuda.synchronize()
    sc, bi = _bn(net)
    kinds = [r[0] for r in rec]
    assert kinds.count("conv") == 53 and kinds.count("maxpool") == 1
    for kind, key, inp, out, res in rec:
        if kind == "conv":
            L = net.layers[key]
            print(f"[resnet50] {L.name}: {tuple(inp.shape)} -> {tuple(out.shape)}", flush=True)
            x = inp.float().cpu().numpy()
            r = None if res is None else res.float().cpu().numpy().reshape(-1, L.Cout)
            y, yabs = orn.conv_layer(x, L, ws[key], net.G, sc[key], bi[key], residual=r, want_abs=True)
            got = out.float().cpu().numpy().reshape(-1, L.Cout)
            assert got.shape == y.shape
            check_close(got, y, epilogue_terms(yabs, sc[key], bi[key], r), TOL["bf16"], L.name)
            del x, r, y, yabs, got
        elif kind == "maxpool":
            ref = oracle.maxpool2d_nhwc(inp.float().cpu().numpy(), 3, 2, 1)
            assert np.array_equal(out.float().cpu().numpy(), ref), "maxpool is exact"
        elif kind == "avgpool":
            xin = inp.float().cpu().numpy()
            ref = oracle.global_avgpool_nhwc(xin)
            terms = np.abs(xin).mean(axis=(1, 2))
            check_close(out.float().cpu().numpy(), ref, terms, TOL["bf16"], "avgpool")
        elif kind == "fc":
            pooled = inp.float().cpu().numpy()
            Wfc = orn.masked_weight(fcw, net.G, net.G)
            ref = oracle.dense_rows(pooled, Wfc)
            terms = np.abs(pooled) @ np.abs(Wfc).T
            check_close(out.cpu().numpy(), ref, terms, TOL["bf16"], "fc")
    assert torch.isfinite(logits).all()
