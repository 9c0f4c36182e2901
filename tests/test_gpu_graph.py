"""HIP-graph capture of the hot path (cci_pack + cci_conv_im2col / cci_spmm
on the dense-tile, sparse-MAC, narrow, wide-tile, streaming, tap-chunk and
split-reduction kernels): every replay, with eager work and synchronisation in between,
reproduces the eager results bit for bit (the kernels are deterministic and
the library records no memset or allocation into a captured graph)."""
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
    # a MobileNetV2-shaped 1x1 conv (24 -> 144) on the narrow kernels and a
    # 4096-channel FC product on the wide-tile ones
    Xn = torch.from_numpy(np.random.default_rng(7).standard_normal((2, 15, 13, 24)).astype(np.float32)).to(
        torch.bfloat16).to(DEV)
    Wn = torch.from_numpy((np.random.default_rng(8).standard_normal((144, 24)) / 5).astype(np.float32)).to(DEV)
    vn = torch.empty((18, 3, 24), dtype=torch.bfloat16, device=DEV)
    xn = torch.empty((18, 3, 24), dtype=torch.uint8, device=DEV)
    Yn = torch.empty((2, 15, 13, 144), dtype=torch.bfloat16, device=DEV)
    Xw = torch.from_numpy(np.random.default_rng(9).standard_normal((300, 1024)).astype(np.float32)).to(
        torch.bfloat16).to(DEV)
    Ww = torch.from_numpy((np.random.default_rng(10).standard_normal((256, 1024)) / 32).astype(np.float32)).to(DEV)
    vw = torch.empty((16, 1, 1024), dtype=torch.bfloat16, device=DEV)
    xw = torch.empty((16, 1, 1024), dtype=torch.uint8, device=DEV)
    Yw = torch.empty((300, 256), dtype=torch.bfloat16, device=DEV)
    # a streaming-kernel product with a residual epilogue, and a tap-chunk 3x3 conv over 128 channels
    Xs2 = torch.from_numpy(np.random.default_rng(11).standard_normal((3000, 64)).astype(np.float32)).to(
        torch.bfloat16).to(DEV)
    Ws2 = torch.from_numpy((np.random.default_rng(12).standard_normal((256, 64)) / 8).astype(np.float32)).to(DEV)
    Rs2 = torch.from_numpy(np.random.default_rng(13).standard_normal((3000, 256)).astype(np.float32)).to(
        torch.bfloat16).to(DEV)
    vs2 = torch.empty((32, 2, 64), dtype=torch.bfloat16, device=DEV)
    xs2 = torch.empty((32, 2, 64), dtype=torch.uint8, device=DEV)
    Ys2 = torch.empty((3000, 256), dtype=torch.bfloat16, device=DEV)
    Xt = torch.from_numpy(np.random.default_rng(14).standard_normal((2, 9, 11, 128)).astype(np.float32)).to(
        torch.bfloat16).to(DEV)
    Wt = torch.from_numpy((np.random.default_rng(15).standard_normal((128, 9 * 128)) / 34).astype(np.float32)).to(DEV)
    vt = torch.empty((16, 2, 9 * 128), dtype=torch.bfloat16, device=DEV)
    xt = torch.empty((16, 2, 9 * 128), dtype=torch.uint8, device=DEV)
    Yt = torch.empty((2, 9, 11, 128), dtype=torch.bfloat16, device=DEV)
    # a split-reduction product (MobileNetV2's 960 -> 160 projection at 7 x 7, one image) with a scale
    Xk = torch.from_numpy(np.random.default_rng(16).standard_normal((49, 960)).astype(np.float32)).to(
        torch.bfloat16).to(DEV)
    Wk = torch.from_numpy((np.random.default_rng(17).standard_normal((160, 960)) / 31).astype(np.float32)).to(DEV)
    Sk = torch.from_numpy(np.random.default_rng(18).uniform(0.5, 1.5, 160).astype(np.float32)).to(DEV)
    vk = torch.empty((20, 2, 960), dtype=torch.bfloat16, device=DEV)
    xk = torch.empty((20, 2, 960), dtype=torch.uint8, device=DEV)
    Yk = torch.empty((49, 160), dtype=torch.bfloat16, device=DEV)
    s = torch.cuda.Stream()

    def step():
        cci.pack(W, w.G, w.K, torch.bfloat16, out=(vals, idx))
        for i in range(3):
            cci.conv_im2col(Xs[i], vals, idx, w.G, 3, 3, (1, 1), (1, 1), out=Ys[i])
        cci.pack(Wf, 8, 4, torch.float32, out=(vf, xf))
        cci.spmm(Xf, vf, xf, 8, out=Yf)
        cci.pack(Wn, 8, 3, torch.bfloat16, out=(vn, xn))
        cci.conv_im2col(Xn, vn, xn, 8, 1, 1, out=Yn, algo="narrow_mfma")
        cci.pack(Ww, 16, 1, torch.bfloat16, out=(vw, xw))
        cci.spmm(Xw, vw, xw, 16, out=Yw, algo="wide_tile_mfma")
        cci.pack(Ws2, 8, 2, torch.bfloat16, out=(vs2, xs2))
        cci.spmm(Xs2, vs2, xs2, 8, residual=Rs2, relu=True, out=Ys2, algo="stream_tile_mfma")
        cci.pack(Wt, 8, 2, torch.bfloat16, out=(vt, xt))
        cci.conv_im2col(Xt, vt, xt, 8, 3, 3, (1, 1), (1, 1), out=Yt, algo="tap_tile_mfma")
        cci.pack(Wk, 8, 2, torch.bfloat16, out=(vk, xk))
        cci.spmm(Xk, vk, xk, 8, scale=Sk, out=Yk, algo="split_k_mfma")

    with torch.cuda.stream(s):
        step()
    torch.cuda.synchronize()
    ref = [y.clone() for y in Ys] + [Yf.clone(), vals.clone(), idx.clone(), Yn.clone(), Yw.clone(), Ys2.clone(),
                                     Yt.clone(), Yk.clone()]

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        step()
    for rep in range(4):
        for y in Ys:
            y.zero_()
        Yf.zero_()
        Yn.zero_()
        Yw.zero_()
        Ys2.zero_()
        Yt.zero_()
        Yk.zero_()
        vals.zero_()
        torch.cuda.synchronize()
        with torch.cuda.stream(s):
            g.replay()
        torch.cuda.synchronize()
        got = Ys + [Yf, vals, idx, Yn, Yw, Ys2, Yt, Yk]
        for a, b in zip(got, ref):
            assert torch.equal(a, b), f"replay {rep} differs from the eager run"
        # eager work between replays, on other data
        tmp = cci.conv_im2col(Xs[2], vals, idx, w.G, 3, 3, (1, 1), (1, 1))
        torch.cuda.synchronize()
        assert torch.equal(tmp, ref[2])
