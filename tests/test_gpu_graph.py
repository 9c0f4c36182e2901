"""HIP-graph capture of the hot path (cci_pack + cci_conv_im2col / cci_spmm):
every replay, with eager work and synchronisation in between, reproduces the
eager results bit for bit (the kernels are deterministic and the library
records no memset or allocation into a captured graph)."""
import numpy as np
import pytest
import torch

from gpu_common import DEV, need_gpu
from paper_1910_11971_amd import cci, workloads as wl

pytestmark = pytest.mark.gpu


def test_graph_replays_match_eager():
    need_gpu()
    w = wl.small(wl.WORKLOADS["conv3x3"], B=3, H=20, W=23)
    X_cpu, W_np = wl.draw(w)
    Xs = [(X_cpu.float() * (1 + 0.25 * i)).to(torch.bfloat16).to(DEV) for i in range(3)]
    W = torch.from_numpy(W_np).to(DEV)
    vals = torch.empty((w.O // w.G, w.K, w.C), dtype=torch.bfloat16, device=DEV)
    idx = torch.empty((w.O // w.G, w.K, w.C), dtype=torch.uint8, device=DEV)
    Ys = [torch.empty((w.B, w.Ho, w.Wo, w.O), dtype=torch.bfloat16, device=DEV) for _ in range(3)]
    Xf = torch.from_numpy(np.random.default_rng(5).standard_normal((64, 256)).astype(np.float32)).to(DEV)
    Wf = torch.from_numpy((np.random.default_rng(6).standard_normal((128, 256)) / 16).astype(np.float32)).to(DEV)
    vf = torch.empty((16, 4, 256), dtype=torch.float32, device=DEV)
    xf = torch.empty((16, 4, 256), dtype=torch.uint8, device=DEV)
    Yf = torch.empty((64, 128), dtype=torch.float32, device=DEV)
    s = torch.cuda.Stream()

    def step():
        cci.pack(W, w.G, w.K, torch.bfloat16, out=(vals, idx))
        for i in range(3):
            cci.conv_im2col(Xs[i], vals, idx, w.G, 3, 3, (1, 1), (1, 1), out=Ys[i])
        cci.pack(Wf, 8, 4, torch.float32, out=(vf, xf))
        cci.spmm(Xf, vf, xf, 8, out=Yf)

    with torch.cuda.stream(s):
        step()
    torch.cuda.synchronize()
    ref = [y.clone() for y in Ys] + [Yf.clone(), vals.clone(), idx.clone()]

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        step()
    for rep in range(4):
        for y in Ys:
            y.zero_()
        Yf.zero_()
        vals.zero_()
        torch.cuda.synchronize()
        with torch.cuda.stream(s):
            g.replay()
        torch.cuda.synchronize()
        got = Ys + [Yf, vals, idx]
        for a, b in zip(got, ref):
            assert torch.equal(a, b), f"replay {rep} differs from the eager run"
        # eager work between replays, on other data
        tmp = cci.conv_im2col(Xs[2], vals, idx, w.G, 3, 3, (1, 1), (1, 1))
        torch.cuda.synchronize()
        assert torch.equal(tmp, ref[2])
