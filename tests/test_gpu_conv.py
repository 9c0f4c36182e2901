"""cci_conv_im2col on the GPU vs the oracle's direct convolution."""
import numpy as np
import pytest
import torch

import oracle
from gpu_common import (DEV, Guarded, epilogue_terms, need_gpu, oracle_pack_vals, rand_epilogue, tol_for,
                        x_as_f32)
from parity import check_close, to_np_f32
from paper_1910_11971_amd import workloads

pytestmark = pytest.mark.gpu


def run_conv(X: torch.Tensor, W: np.ndarray, G, K, k, stride, pad, y_dtype, algo, *, pixels=None,
             ep=None):
    return run_conv_kw(X, W, G, K, k, k, stride, pad, y_dtype, algo, pixels=pixels, ep=ep)


def run_conv_kw(X: torch.Tensor, W: np.ndarray, G, K, KH, KW, stride, pad, y_dtype, algo, *, pixels=None,
                ep=None):
    from paper_1910_11971_amd import cci
    vdt = torch.float32 if X.dtype == torch.float32 else torch.bfloat16
    B, H, Wd, Cin = X.shape
    O = W.shape[0]
    s, b, r, r_t, relu = ep if ep is not None else (None, None, None, None, False)
    kw = {}
    if s is not None:
        kw["scale"] = torch.from_numpy(s).to(DEV)
    if b is not None:
        kw["bias"] = torch.from_numpy(b).to(DEV)
    Ho, Wo = cci.conv_out_hw(H, Wd, KH, KW, (stride, stride), (pad, pad))
    if r_t is not None:
        kw["residual"] = r_t.reshape(B, Ho, Wo, O).to(DEV)
    vals, idx = cci.pack(torch.from_numpy(W).to(DEV), G, K, vdt)
    Yg = Guarded((B, Ho, Wo, O), y_dtype)
    Y = cci.conv_im2col(X.to(DEV), vals, idx, G, KH, KW, (stride, stride), (pad, pad), relu=relu,
                        out_dtype=y_dtype, algo=algo, out=Yg.t, **kw)
    torch.cuda.synchronize()
    Yg.check(f"conv {algo} {tuple(X.shape)} k{KH}x{KW} s{stride} p{pad} O={O}")
    v_ref, idx_ref, _ = oracle_pack_vals(W, G, K, vdt)
    Wmask = oracle.unpack(v_ref, idx_ref, G).reshape(O, KH, KW, Cin)
    Yref, Yabs = oracle.conv2d_nhwc(x_as_f32(X), Wmask, (stride, stride), (pad, pad), scale=s, bias=b,
                                    residual=r, relu=relu, pixels=pixels, want_abs=True)
    got = to_np_f32(Y).reshape(-1, O)
    if pixels is not None:
        got = got[pixels]
    rr = None if r is None else (r if pixels is None else r[pixels])
    S = epilogue_terms(Yabs, s, b, rr)
    return check_close(got, Yref, S, tol_for(y_dtype, X.dtype),
                       f"conv {algo} {tuple(X.shape)} k{KH}x{KW} s{stride} p{pad} O={O} G={G} K={K}")


def rand_x(shape, dtype, seed):
    return torch.from_numpy(np.random.default_rng(seed).standard_normal(shape).astype(np.float32)).to(dtype)


def rand_w(O, C, seed):
    return (np.random.default_rng(seed).standard_normal((O, C)) / np.sqrt(C)).astype(np.float32)


CASES = [  # B, H, W, Cin, O, k, stride, pad, G, K
    (2, 9, 11, 32, 64, 3, 1, 1, 8, 2),
    (3, 14, 14, 64, 64, 3, 2, 1, 8, 2),
    (2, 7, 7, 64, 128, 1, 1, 0, 16, 4),
    (2, 13, 10, 32, 64, 1, 2, 0, 8, 3),
    (1, 6, 5, 96, 64, 3, 1, 0, 4, 1),
    (4, 17, 19, 32, 192, 3, 2, 1, 16, 2),
]


@pytest.mark.parametrize("algo", ["sparse_mac", "dense_tile_mfma"])
@pytest.mark.parametrize("B,H,W,Cin,O,k,stride,pad,G,K", CASES)
def test_conv_bf16(B, H, W, Cin, O, k, stride, pad, G, K, algo):
    need_gpu()
    X = rand_x((B, H, W, Cin), torch.bfloat16, B * H + Cin)
    run_conv(X, rand_w(O, k * k * Cin, O + k), G, K, k, stride, pad, torch.bfloat16, algo)


@pytest.mark.parametrize("B,H,W,Cin,O,G,K", [(2, 14, 14, 128, 256, 16, 4), (3, 9, 13, 64, 512, 8, 2)])
def test_conv1x1_wide_tile(B, H, W, Cin, O, G, K):
    """Stride-1 unpadded 1x1 convolution on the wide-tile kernels (pixels are X rows)."""
    need_gpu()
    X = rand_x((B, H, W, Cin), torch.bfloat16, B * H + Cin)
    ep = rand_epilogue(O, B * H * W, torch.bfloat16, 8, residual=True, relu=True)
    run_conv(X, rand_w(O, Cin, O + 1), G, K, 1, 1, 0, torch.bfloat16, "wide_tile_mfma", ep=ep)


NARROW_CONV_CASES = [  # B, H, W, Cin, O, KH, KW, stride, pad, G, K
    (1, 40, 38, 4, 64, 7, 8, 2, 3, 8, 8),     # a first conv: 3 channels padded to 4, 7x7 padded to 7x8
    (2, 21, 17, 4, 64, 7, 8, 2, 3, 8, 2),
    (2, 9, 11, 4, 32, 3, 4, 1, 1, 8, 3),
    (2, 13, 10, 8, 64, 3, 3, 1, 1, 8, 2),
    (3, 14, 15, 16, 96, 3, 3, 2, 1, 16, 5),
    (1, 12, 12, 24, 48, 3, 3, 1, 0, 8, 1),
    (2, 6, 7, 8, 16, 5, 5, 1, 2, 4, 4),
    (2, 10, 9, 40, 24, 1, 1, 2, 0, 8, 2),     # strided 1x1
]


@pytest.mark.parametrize("B,H,W,Cin,O,KH,KW,stride,pad,G,K", NARROW_CONV_CASES)
def test_conv_narrow_implicit_im2col(B, H, W, Cin, O, KH, KW, stride, pad, G, K):
    need_gpu()
    from paper_1910_11971_amd import cci
    X = rand_x((B, H, W, Cin), torch.bfloat16, Cin + O + KH)
    W_ = rand_w(O, KH * KW * Cin, O + KW)
    Ho, Wo = cci.conv_out_hw(H, W, KH, KW, (stride, stride), (pad, pad))
    ep = rand_epilogue(O, B * Ho * Wo, torch.bfloat16, 6, residual=True, relu=True)
    run_conv_kw(X, W_, G, K, KH, KW, stride, pad, torch.bfloat16, "narrow_mfma", ep=ep)


@pytest.mark.parametrize("B,H,W,Cin,O,G,K", [(2, 7, 9, 24, 144, 8, 3), (3, 11, 5, 144, 32, 8, 1),
                                             (1, 28, 28, 16, 96, 8, 2)])
def test_conv1x1_narrow(B, H, W, Cin, O, G, K):
    need_gpu()
    X = rand_x((B, H, W, Cin), torch.bfloat16, Cin + O)
    ep = rand_epilogue(O, B * H * W, torch.bfloat16, 5, relu=True)
    run_conv(X, rand_w(O, Cin, O), G, K, 1, 1, 0, torch.bfloat16, "narrow_mfma", ep=ep)


RESIDENT_CASES = [  # B, H, W, Cin, O, pad, G, K
    (2, 9, 11, 32, 64, 1, 8, 2),
    (3, 14, 14, 64, 64, 1, 8, 2),
    (1, 6, 5, 64, 32, 0, 4, 1),      # 32 outputs: eight pixel streams; no padding
    (2, 17, 19, 32, 32, 2, 16, 5),   # padding 2
    (5, 12, 23, 64, 64, 1, 64, 64),  # K = G (dense control): 4608 packed units
    (3, 3, 3, 64, 64, 1, 32, 7),     # a 3x3 image: one band of 3 rows
    (1, 5, 100, 64, 64, 1, 2, 1),    # 16 KiB staged rows
    (2, 7, 120, 32, 64, 0, 4, 2),    # 16 KiB staged rows, 32 channels
    (7, 31, 13, 32, 64, 1, 1, 1),    # G = 1
    (9, 10, 10, 64, 64, 1, 8, 3),    # 18 bands: not a multiple of 8 (no XCD grouping)
]


@pytest.mark.parametrize("B,H,W,Cin,O,pad,G,K", RESIDENT_CASES)
def test_conv_resident(B, H, W, Cin, O, pad, G, K):
    """3x3 unit-stride convolutions on the register-resident kernels."""
    need_gpu()
    X = rand_x((B, H, W, Cin), torch.bfloat16, B + H + W + Cin)
    run_conv(X, rand_w(O, 9 * Cin, O + G + K), G, K, 3, 1, pad, torch.bfloat16, "resident_mfma")


@pytest.mark.parametrize("y_dtype", [torch.bfloat16, torch.float32])
@pytest.mark.parametrize("O", [32, 64])
def test_conv_resident_epilogue(y_dtype, O):
    """scale, bias, residual and ReLU fused on the resident kernels, bf16 and fp32 output."""
    need_gpu()
    B, H, W, Cin = 3, 11, 13, 64
    ep = rand_epilogue(O, B * H * W, y_dtype, O + 3, residual=True, relu=True)
    run_conv(rand_x((B, H, W, Cin), torch.bfloat16, 41), rand_w(O, 9 * Cin, 42), 8, 2, 3, 1, 1, y_dtype,
             "resident_mfma", ep=ep)
    ep = rand_epilogue(O, B * H * W, y_dtype, O + 4, residual=False, relu=False)
    run_conv(rand_x((B, H, W, Cin), torch.bfloat16, 43), rand_w(O, 9 * Cin, 44), 8, 2, 3, 1, 1, y_dtype,
             "resident_mfma", ep=ep)


def test_conv_resident_wide_rows_fall_back():
    """Rows wider than 16 KiB of staged activations are refused by the resident family and run under AUTO."""
    need_gpu()
    from paper_1910_11971_amd import cci
    X = rand_x((1, 4, 200, 64), torch.bfloat16, 61)
    vals, idx = cci.pack(torch.from_numpy(rand_w(64, 576, 62)).to(DEV), 8, 2, torch.bfloat16)
    with pytest.raises(cci.CCIError):
        cci.conv_im2col(X.to(DEV), vals, idx, 8, 3, 3, (1, 1), (1, 1), algo="resident_mfma")
    run_conv(X, rand_w(64, 576, 62), 8, 2, 3, 1, 1, torch.bfloat16, "auto")


def test_conv_resident_is_auto_for_3x3_64():
    from paper_1910_11971_amd import cci
    assert cci.auto_algo(torch.bfloat16, torch.bfloat16, 100352, 576, 64, 64, 8, 2) == "resident_mfma"


@pytest.mark.parametrize("stride", [2])
def test_conv_resident_shape_falls_back(stride):
    """A strided 3x3 64 -> 64 layer (not a resident shape) still runs under AUTO."""
    need_gpu()
    X = rand_x((2, 15, 15, 64), torch.bfloat16, 51)
    run_conv(X, rand_w(64, 576, 52), 8, 2, 3, stride, 1, torch.bfloat16, "auto")


TAP_CASES = [  # B, H, W, Cin, O, KH, KW, stride, pad, G, K
    (2, 9, 11, 64, 128, 3, 3, 1, 1, 8, 2),     # 198 pixels: a ragged second pixel block
    (3, 14, 14, 128, 128, 3, 3, 2, 1, 8, 2),   # stride 2
    (2, 7, 7, 256, 256, 3, 3, 1, 1, 16, 4),    # one pixel block, two output blocks, 36 chunks
    (1, 12, 10, 64, 384, 5, 5, 1, 2, 4, 1),    # 5x5, padding 2, three output blocks
    (2, 10, 9, 128, 128, 1, 1, 2, 0, 16, 2),   # strided 1x1
    (3, 8, 8, 64, 128, 3, 3, 1, 0, 32, 7),     # G = 32: a group spans two 16-row blocks
    (2, 6, 7, 64, 128, 3, 3, 1, 1, 8, 8),      # K = G (dense control)
    (4, 9, 9, 64, 256, 3, 3, 2, 1, 2, 1),      # G = 2: 16 packed rows per wave
    (2, 11, 13, 192, 128, 3, 3, 1, 1, 8, 3),   # 12 packed rows per wave; 3 channel blocks per tap
    (1, 20, 20, 64, 128, 7, 4, 1, 3, 16, 1),   # 28 taps, padding 3
    (6, 16, 16, 64, 128, 1, 1, 1, 0, 4, 2),    # 1x1 through the conv call; 16 packed rows per wave
    (3, 4, 4, 64, 128, 3, 3, 1, 1, 1, 1),      # G = 1
    (1, 1, 1, 64, 128, 3, 3, 1, 1, 8, 2),      # one pixel: every tap but the centre in the padding
    (10, 60, 60, 64, 128, 3, 3, 1, 1, 8, 2),   # 282 workgroups: two per CU
    (4, 30, 30, 128, 256, 3, 3, 1, 1, 16, 4),  # 226 workgroups: one per CU
    (2, 9, 11, 64, 64, 3, 3, 1, 1, 8, 2),      # 64 outputs: 64-output tiles
    (3, 14, 14, 128, 192, 3, 3, 2, 1, 16, 4),  # 192 outputs: three 64-output tiles
    (16, 28, 28, 64, 64, 3, 3, 1, 1, 8, 2),    # 98 pixel blocks x 1: 64-output tiles, one per CU
    (40, 28, 28, 64, 64, 3, 3, 2, 1, 4, 2),    # 245 pixel blocks of 64-output tiles
    (12, 40, 40, 64, 320, 1, 1, 1, 0, 16, 8),  # 150 x 5 = 750 tiles of 64 outputs: two per CU
]


@pytest.mark.parametrize("B,H,W,Cin,O,KH,KW,stride,pad,G,K", TAP_CASES)
def test_conv_tap_tile(B, H, W, Cin, O, KH, KW, stride, pad, G, K):
    """Implicit-im2col convolutions on the tap-chunk kernels (128 x 128 tiles)."""
    need_gpu()
    X = rand_x((B, H, W, Cin), torch.bfloat16, B + H + W + Cin + KH)
    run_conv_kw(X, rand_w(O, KH * KW * Cin, O + G + K + KW), G, K, KH, KW, stride, pad, torch.bfloat16,
                "tap_tile_mfma")


@pytest.mark.parametrize("y_dtype", [torch.bfloat16, torch.float32])
def test_conv_tap_tile_epilogue(y_dtype):
    """scale, bias, residual and ReLU fused on the tap-chunk kernels, bf16 and fp32 output."""
    need_gpu()
    from paper_1910_11971_amd import cci
    B, H, W, Cin, O = 2, 13, 11, 128, 256
    Ho, Wo = cci.conv_out_hw(H, W, 3, 3, (2, 2), (1, 1))
    ep = rand_epilogue(O, B * Ho * Wo, y_dtype, 71, residual=True, relu=True)
    run_conv(rand_x((B, H, W, Cin), torch.bfloat16, 72), rand_w(O, 9 * Cin, 73), 8, 2, 3, 2, 1, y_dtype,
             "tap_tile_mfma", ep=ep)
    ep = rand_epilogue(O, B * Ho * Wo, y_dtype, 74, residual=False, relu=False)
    run_conv(rand_x((B, H, W, Cin), torch.bfloat16, 75), rand_w(O, 9 * Cin, 76), 16, 4, 3, 2, 1, y_dtype,
             "tap_tile_mfma", ep=ep)


def test_conv_tap_tile_refuses_unsupported():
    """Cin % 64 != 0, O % 64 != 0, G = 64, and G = 32 with O % 128 != 0 are refused by the tap-chunk family."""
    need_gpu()
    from paper_1910_11971_amd import cci
    for Cin, O, G in [(96, 128, 8), (64, 96, 8), (64, 128, 64), (64, 192, 32)]:
        X = rand_x((1, 5, 5, Cin), torch.bfloat16, 81).to(DEV)
        vals, idx = cci.pack(torch.from_numpy(rand_w(O, 9 * Cin, 82)).to(DEV), G, 2, torch.bfloat16)
        with pytest.raises(cci.CCIError):
            cci.conv_im2col(X, vals, idx, G, 3, 3, (1, 1), (1, 1), algo="tap_tile_mfma")


@pytest.mark.parametrize("B,H,W,Cin,O,G,K,y_dtype", [(4, 30, 30, 128, 256, 8, 2, torch.bfloat16),
                                                     (3, 17, 13, 64, 192, 16, 4, torch.float32),
                                                     (2, 28, 28, 256, 64, 8, 2, torch.bfloat16)])
def test_conv_stream_tile_1x1(B, H, W, Cin, O, G, K, y_dtype):
    """1x1 stride-1 convolutions on the streaming kernels, every epilogue term."""
    need_gpu()
    ep = rand_epilogue(O, B * H * W, y_dtype, 91 + Cin, residual=True, relu=True)
    run_conv(rand_x((B, H, W, Cin), torch.bfloat16, 92 + O), rand_w(O, Cin, 93 + G), G, K, 1, 1, 0, y_dtype,
             "stream_tile_mfma", ep=ep)


def test_conv_stream_tile_refuses_unsupported():
    """3x3, strided or padded 1x1 convolutions are not streaming-kernel products."""
    need_gpu()
    from paper_1910_11971_amd import cci
    for k, stride, pad in [(3, 1, 1), (1, 2, 0), (1, 1, 1)]:
        X = rand_x((1, 9, 9, 64), torch.bfloat16, 95).to(DEV)
        vals, idx = cci.pack(torch.from_numpy(rand_w(128, k * k * 64, 96)).to(DEV), 8, 2, torch.bfloat16)
        with pytest.raises(cci.CCIError):
            cci.conv_im2col(X, vals, idx, 8, k, k, (stride, stride), (pad, pad), algo="stream_tile_mfma")


@pytest.mark.parametrize("B,H,W,Cin,O,G,K,y_dtype", [(64, 7, 7, 960, 160, 8, 2, torch.bfloat16),
                                                     (5, 14, 14, 384, 64, 8, 3, torch.float32),
                                                     (3, 9, 11, 576, 96, 16, 4, torch.bfloat16)])
def test_conv_split_k_1x1(B, H, W, Cin, O, G, K, y_dtype):
    """1x1 stride-1 convolutions on the split-reduction kernels, every epilogue term."""
    need_gpu()
    ep = rand_epilogue(O, B * H * W, y_dtype, 97 + Cin, residual=True, relu=True)
    run_conv(rand_x((B, H, W, Cin), torch.bfloat16, 98 + O), rand_w(O, Cin, 99 + G), G, K, 1, 1, 0, y_dtype,
             "split_k_mfma", ep=ep)


def test_conv_split_k_refuses_unsupported():
    """3x3, strided or padded 1x1 convolutions are not split-reduction products."""
    need_gpu()
    from paper_1910_11971_amd import cci
    for k, stride, pad in [(3, 1, 1), (1, 2, 0), (1, 1, 1)]:
        X = rand_x((1, 9, 9, 64), torch.bfloat16, 95).to(DEV)
        vals, idx = cci.pack(torch.from_numpy(rand_w(128, k * k * 64, 96)).to(DEV), 8, 2, torch.bfloat16)
        with pytest.raises(cci.CCIError):
            cci.conv_im2col(X, vals, idx, 8, k, k, (stride, stride), (pad, pad), algo="split_k_mfma")


@pytest.mark.parametrize("algo", ["sparse_mac", "dense_tile_mfma"])
def test_conv_epilogue_residual_relu(algo):
    need_gpu()
    B, H, W, Cin, O, k = 2, 10, 10, 64, 64, 3
    N = B * H * W
    ep = rand_epilogue(O, N, torch.bfloat16, 11, residual=True, relu=True)
    run_conv(rand_x((B, H, W, Cin), torch.bfloat16, 12), rand_w(O, k * k * Cin, 13), 8, 2, k, 1, 1,
             torch.bfloat16, algo, ep=ep)


def test_conv_stem_7x7_cin3_dense_control():
    """ResNet stem shape: 7x7 stride 2 pad 3, Cin=3 (K=G: dense control)."""
    need_gpu()
    X = rand_x((2, 32, 32, 3), torch.bfloat16, 21)
    run_conv(X, rand_w(64, 147, 22), 8, 8, 7, 2, 3, torch.bfloat16, "auto")


def test_conv_fp32():
    need_gpu()
    X = rand_x((2, 8, 8, 5), torch.float32, 31)
    run_conv(X, rand_w(16, 45, 32), 4, 2, 3, 1, 1, torch.float32, "auto")
