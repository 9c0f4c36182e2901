"""CPU-only checks of the C ABI: the library loads, exports every function
include/cci.h declares, and rejects bad arguments before touching the GPU."""
import ctypes

import pytest
import torch

from paper_1910_11971_amd import cci

lib = cci.raw()
FAKE = ctypes.c_void_p(0x10000)          # aligned, never dereferenced: validation fails first
FAKE_MIS = ctypes.c_void_p(0x10008)      # 8-byte aligned only


def test_exports_every_declared_symbol():
    names = cci.header_functions()
    assert {"cci_pack", "cci_spmm", "cci_conv_im2col", "cci_packed_sizes", "cci_spmm_algo",
            "cci_conv_im2col_algo"} <= set(names)
    for n in names:
        assert hasattr(lib, n), f"libcci.so does not export {n}"
    assert cci.version() >= 100


def test_packed_sizes_arithmetic():
    assert cci.packed_sizes(256, 256, 8, 4, torch.float32) == (256 // 8 * 4 * 256 * 4, 256 // 8 * 4 * 256)
    assert cci.packed_sizes(64, 576, 8, 2, torch.bfloat16) == (8 * 2 * 576 * 2, 8 * 2 * 576)
    vb, ib = cci.packed_sizes(4096, 4096, 16, 1)
    assert ib == 4096 * 4096 // 16 and vb == 2 * ib


@pytest.mark.parametrize("O,C,G,K", [(12, 5, 8, 2), (16, 5, 8, 0), (16, 5, 8, 9), (16, 0, 8, 2),
                                     (512, 5, 512, 2), (16, 5, 0, 1)])
def test_bad_group_arguments(O, C, G, K):
    vb, ib = ctypes.c_size_t(77), ctypes.c_size_t(77)
    assert lib.cci_packed_sizes(O, C, G, K, cci.BF16, ctypes.byref(vb), ctypes.byref(ib)) == cci.EINVAL
    assert vb.value == 77 and ib.value == 77           # outputs untouched
    assert lib.cci_last_error()
    assert lib.cci_pack(FAKE, O, C, G, K, FAKE, cci.BF16, FAKE, None) == cci.EINVAL
    assert lib.cci_spmm(FAKE, cci.BF16, 4, C, FAKE, cci.BF16, FAKE, O, G, K, None, FAKE,
                        cci.BF16, None) == cci.EINVAL


def test_null_and_alignment_errors():
    assert lib.cci_pack(None, 16, 8, 8, 2, FAKE, cci.F32, FAKE, None) == cci.EINVAL
    assert lib.cci_pack(FAKE_MIS, 16, 8, 8, 2, FAKE, cci.F32, FAKE, None) == cci.EALIGN
    assert lib.cci_spmm(FAKE, cci.F32, 4, 8, FAKE, cci.F32, FAKE, 16, 8, 2, None, None,
                        cci.F32, None) == cci.EINVAL
    assert lib.cci_spmm(FAKE, cci.F32, 4, 8, FAKE, cci.F32, FAKE_MIS, 16, 8, 2, None, FAKE,
                        cci.F32, None) == cci.EALIGN
    ep = cci.Epilogue(ctypes.c_void_p(0x10004), None, None, 0)
    assert lib.cci_spmm(FAKE, cci.F32, 4, 8, FAKE, cci.F32, FAKE, 16, 8, 2, ctypes.byref(ep),
                        FAKE, cci.F32, None) == cci.EALIGN
    assert "align" in lib.cci_last_error().decode()


def test_dtype_combinations():
    # f32 X with bf16 values, bf16 X with f32 values: unsupported
    assert lib.cci_spmm(FAKE, cci.F32, 4, 8, FAKE, cci.BF16, FAKE, 16, 8, 2, None, FAKE,
                        cci.F32, None) == cci.EUNSUPPORTED
    assert lib.cci_spmm(FAKE, cci.BF16, 4, 8, FAKE, cci.F32, FAKE, 16, 8, 2, None, FAKE,
                        cci.BF16, None) == cci.EUNSUPPORTED
    assert lib.cci_spmm(FAKE, cci.F32, 4, 8, FAKE, cci.F32, FAKE, 16, 8, 2, None, FAKE,
                        cci.BF16, None) == cci.EUNSUPPORTED
    assert lib.cci_spmm(FAKE, 7, 4, 8, FAKE, cci.F32, FAKE, 16, 8, 2, None, FAKE,
                        cci.F32, None) == cci.EINVAL


def test_explicit_algo_requirements():
    # dense-tile MFMA needs bf16 and C % 32 == 0; sparse-MAC needs G in {2,4,8,16,32}
    assert lib.cci_spmm_algo(FAKE, cci.F32, 4, 64, FAKE, cci.F32, FAKE, 16, 8, 2, None, FAKE,
                        cci.F32, cci.ALGO_DENSE_TILE_MFMA, None) == cci.EUNSUPPORTED
    assert lib.cci_spmm_algo(FAKE, cci.BF16, 4, 40, FAKE, cci.BF16, FAKE, 16, 8, 2, None, FAKE,
                        cci.BF16, cci.ALGO_DENSE_TILE_MFMA, None) == cci.EUNSUPPORTED
    assert lib.cci_spmm_algo(FAKE, cci.BF16, 4, 64, FAKE, cci.BF16, FAKE, 24, 6, 2, None, FAKE,
                        cci.BF16, cci.ALGO_SPARSE_MAC, None) == cci.EUNSUPPORTED
    assert lib.cci_spmm_algo(FAKE, cci.BF16, 4, 64, FAKE, cci.BF16, FAKE, 16, 8, 2, None, FAKE,
                        cci.BF16, 10, None) == cci.EINVAL
    # wide-tile MFMA: O % 256, C % 64, 64 % G, bf16 only; strided / padded / k x k convs refused
    W = cci.ALGO_WIDE_TILE_MFMA
    assert lib.cci_spmm_algo(FAKE, cci.BF16, 4, 64, FAKE, cci.BF16, FAKE, 128, 8, 2, None, FAKE,
                        cci.BF16, W, None) == cci.EUNSUPPORTED
    assert lib.cci_spmm_algo(FAKE, cci.BF16, 4, 96, FAKE, cci.BF16, FAKE, 256, 8, 2, None, FAKE,
                        cci.BF16, W, None) == cci.EUNSUPPORTED
    assert lib.cci_spmm_algo(FAKE, cci.F32, 4, 64, FAKE, cci.F32, FAKE, 256, 8, 2, None, FAKE,
                        cci.F32, W, None) == cci.EUNSUPPORTED
    assert lib.cci_spmm_algo(FAKE, cci.BF16, 4, 64, FAKE, cci.BF16, FAKE, 256, 128, 2, None, FAKE,
                        cci.BF16, W, None) == cci.EUNSUPPORTED
    for KH, sh, ph in [(3, 1, 1), (1, 2, 0), (1, 1, 1)]:
        assert lib.cci_conv_im2col_algo(FAKE, cci.BF16, 1, 8, 8, 64, KH, KH, sh, sh, ph, ph, FAKE, cci.BF16,
                                   FAKE, 256, 8, 2, None, FAKE, cci.BF16, W, None) == cci.EUNSUPPORTED


def test_narrow_algo_requirements():
    # narrow MFMA: bf16, C <= 256, C % 8 == 0, O % 4 == 0; strided / padded / k x k convs refused
    Nw = cci.ALGO_NARROW_MFMA
    assert lib.cci_spmm_algo(FAKE, cci.BF16, 4, 264, FAKE, cci.BF16, FAKE, 16, 8, 2, None, FAKE,
                        cci.BF16, Nw, None) == cci.EUNSUPPORTED
    assert lib.cci_spmm_algo(FAKE, cci.BF16, 4, 20, FAKE, cci.BF16, FAKE, 16, 8, 2, None, FAKE,
                        cci.BF16, Nw, None) == cci.EUNSUPPORTED
    assert lib.cci_spmm_algo(FAKE, cci.BF16, 4, 16, FAKE, cci.BF16, FAKE, 18, 2, 1, None, FAKE,
                        cci.BF16, Nw, None) == cci.EUNSUPPORTED
    assert lib.cci_spmm_algo(FAKE, cci.F32, 4, 16, FAKE, cci.F32, FAKE, 16, 8, 2, None, FAKE,
                        cci.F32, Nw, None) == cci.EUNSUPPORTED
    # convs: Cin 3, Cin 4 with an odd KW, and a reduction past 256 are refused
    for Cin, KH, KW in [(3, 3, 3), (4, 7, 7), (40, 3, 3)]:
        assert lib.cci_conv_im2col_algo(FAKE, cci.BF16, 1, 8, 8, Cin, KH, KW, 1, 1, 1, 1, FAKE, cci.BF16,
                                   FAKE, 96, 8, 2, None, FAKE, cci.BF16, Nw, None) == cci.EUNSUPPORTED


def test_resident_algo_requirements():
    # resident MFMA: bf16 3x3 convolutions with unit stride, Cin 32 / 64, O 32 / 64; FC refused
    Rs = cci.ALGO_RESIDENT_MFMA
    assert lib.cci_spmm_algo(FAKE, cci.BF16, 4, 576, FAKE, cci.BF16, FAKE, 64, 8, 2, None, FAKE,
                             cci.BF16, Rs, None) == cci.EUNSUPPORTED
    for Cin, KH, st, O in [(64, 3, 2, 64), (96, 3, 1, 64), (64, 1, 1, 64), (64, 3, 1, 128), (64, 5, 1, 64),
                           (16, 3, 1, 64)]:
        assert lib.cci_conv_im2col_algo(FAKE, cci.BF16, 1, 8, 8, Cin, KH, KH, st, st, 1, 1, FAKE, cci.BF16,
                                        FAKE, O, 8, 2, None, FAKE, cci.BF16, Rs, None) == cci.EUNSUPPORTED
    assert lib.cci_conv_im2col_algo(FAKE, cci.F32, 1, 8, 8, 64, 3, 3, 1, 1, 1, 1, FAKE, cci.F32,
                                    FAKE, 64, 8, 2, None, FAKE, cci.F32, Rs, None) == cci.EUNSUPPORTED
    # misaligned idx (8-byte alignment needed) -- the plain 16-byte rule fires first
    assert lib.cci_conv_im2col_algo(FAKE, cci.BF16, 1, 8, 8, 64, 3, 3, 1, 1, 1, 1, FAKE, cci.BF16,
                                    FAKE_MIS, 64, 8, 2, None, FAKE, cci.BF16, Rs, None) == cci.EALIGN
    # the shape-only choice names the family for 3x3 64 -> 64
    assert lib.cci_auto_algo(cci.BF16, cci.BF16, 100352, 576, 64, 64, 8, 2) == Rs


def test_tap_tile_algo_requirements():
    # tap-tile MFMA: bf16, Cin (FC: C) % 64 == 0, O % 128 == 0 (O % 64 == 0 with G <= 16), 32 % G == 0,
    # 2 K <= G or K == G, at most 32 taps
    Tt = cci.ALGO_TAP_TILE_MFMA
    for C, O, G, K in [(96, 128, 8, 2), (64, 96, 8, 2), (64, 128, 64, 2), (64, 192, 32, 2), (64, 128, 8, 5)]:
        assert lib.cci_spmm_algo(FAKE, cci.BF16, 4, C, FAKE, cci.BF16, FAKE, O, G, K, None, FAKE,
                                 cci.BF16, Tt, None) == cci.EUNSUPPORTED
    assert lib.cci_spmm_algo(FAKE, cci.F32, 4, 64, FAKE, cci.F32, FAKE, 128, 8, 2, None, FAKE,
                             cci.F32, Tt, None) == cci.EUNSUPPORTED
    for Cin, KH, KW in [(32, 3, 3), (64, 7, 7)]:
        assert lib.cci_conv_im2col_algo(FAKE, cci.BF16, 1, 8, 8, Cin, KH, KW, 1, 1, 1, 1, FAKE, cci.BF16,
                                        FAKE, 128, 8, 2, None, FAKE, cci.BF16, Tt, None) == cci.EUNSUPPORTED


def test_stream_tile_algo_requirements():
    # stream-tile MFMA: bf16, FC or stride-1 unpadded 1x1, C % 64 == 0 with C <= 256, O % 64 == 0, 32 % G == 0
    St = cci.ALGO_STREAM_TILE_MFMA
    for C, O, G, K in [(96, 128, 8, 2), (320, 128, 8, 2), (64, 96, 8, 2), (64, 128, 64, 2)]:
        assert lib.cci_spmm_algo(FAKE, cci.BF16, 4, C, FAKE, cci.BF16, FAKE, O, G, K, None, FAKE,
                                 cci.BF16, St, None) == cci.EUNSUPPORTED
    assert lib.cci_spmm_algo(FAKE, cci.F32, 4, 64, FAKE, cci.F32, FAKE, 128, 8, 2, None, FAKE,
                             cci.F32, St, None) == cci.EUNSUPPORTED
    for k, stride, pad in [(3, 1, 1), (1, 2, 0), (1, 1, 1)]:
        assert lib.cci_conv_im2col_algo(FAKE, cci.BF16, 1, 8, 8, 64, k, k, stride, stride, pad, pad, FAKE, cci.BF16,
                                        FAKE, 128, 8, 2, None, FAKE, cci.BF16, St, None) == cci.EUNSUPPORTED
    assert lib.cci_spmm_algo(FAKE, cci.BF16, 4, 64, FAKE, cci.BF16, FAKE, 128, 8, 2, None, FAKE,
                             cci.BF16, 10, None) == cci.EINVAL


def test_split_k_algo_requirements():
    # split-K MFMA: bf16, FC or stride-1 unpadded 1x1, C % 32 == 0, O % 16 == 0, K <= 4
    Sk = cci.ALGO_SPLIT_K_MFMA
    for C, O, G, K in [(48, 64, 8, 2), (960, 24, 8, 2), (960, 160, 8, 5)]:
        assert lib.cci_spmm_algo(FAKE, cci.BF16, 4, C, FAKE, cci.BF16, FAKE, O, G, K, None, FAKE,
                                 cci.BF16, Sk, None) == cci.EUNSUPPORTED
    assert lib.cci_spmm_algo(FAKE, cci.F32, 4, 960, FAKE, cci.F32, FAKE, 160, 8, 2, None, FAKE,
                             cci.F32, Sk, None) == cci.EUNSUPPORTED
    for k, stride, pad in [(3, 1, 1), (1, 2, 0), (1, 1, 1)]:
        assert lib.cci_conv_im2col_algo(FAKE, cci.BF16, 1, 8, 8, 64, k, k, stride, stride, pad, pad, FAKE, cci.BF16,
                                        FAKE, 128, 8, 2, None, FAKE, cci.BF16, Sk, None) == cci.EUNSUPPORTED


def test_few_rows_algo_requirements():
    # few-row MFMA: bf16 FC / plain 1x1 products with N <= 64, C % 32 == 0, O % 4 == 0
    Fr = cci.ALGO_FEW_ROWS_MFMA
    for N, C, O, G in [(65, 64, 16, 8), (4, 48, 16, 8), (4, 64, 18, 2)]:
        assert lib.cci_spmm_algo(FAKE, cci.BF16, N, C, FAKE, cci.BF16, FAKE, O, G, 2 if G > 2 else 1, None, FAKE,
                                 cci.BF16, Fr, None) == cci.EUNSUPPORTED
    assert lib.cci_spmm_algo(FAKE, cci.F32, 4, 64, FAKE, cci.F32, FAKE, 16, 8, 2, None, FAKE,
                             cci.F32, Fr, None) == cci.EUNSUPPORTED
    assert lib.cci_conv_im2col_algo(FAKE, cci.BF16, 1, 4, 4, 64, 3, 3, 1, 1, 1, 1, FAKE, cci.BF16,
                                    FAKE, 16, 8, 2, None, FAKE, cci.BF16, Fr, None) == cci.EUNSUPPORTED
    assert lib.cci_auto_algo(cci.BF16, cci.BF16, 64, 4096, 4096, 4096, 16, 4) == Fr
    assert lib.cci_auto_algo(cci.BF16, cci.BF16, 65, 4096, 4096, 4096, 16, 4) != Fr
    # a ragged last 16-output tile (the ResNet-50 classifier: 2048 -> 1000) is taken only when pinned
    assert lib.cci_auto_algo(cci.BF16, cci.BF16, 64, 2048, 2048, 1000, 8, 8) != Fr


def test_algo_entry_points_match_plain_calls_on_validation():
    # the pinned-family calls validate exactly like the plain ones
    assert lib.cci_spmm_algo(FAKE, cci.BF16, 4, 64, FAKE, cci.BF16, FAKE, 12, 8, 2, None, FAKE,
                             cci.BF16, cci.ALGO_AUTO, None) == cci.EINVAL
    assert lib.cci_spmm_algo(None, cci.BF16, 0, 64, None, cci.BF16, None, 16, 8, 2, None, None,
                             cci.BF16, cci.ALGO_WIDE_TILE_MFMA, None) == cci.OK
    assert lib.cci_conv_im2col_algo(FAKE, cci.BF16, 1, 5, 5, 32, 3, 3, 0, 1, 1, 1, FAKE, cci.BF16,
                                    FAKE, 16, 8, 2, None, FAKE, cci.BF16, cci.ALGO_AUTO, None) == cci.EINVAL


def test_empty_is_a_noop():
    # N == 0: nothing to do, no pointer is needed or touched
    assert lib.cci_spmm(None, cci.BF16, 0, 64, None, cci.BF16, None, 16, 8, 2, None, None,
                        cci.BF16, None) == cci.OK
    assert lib.cci_conv_im2col(None, cci.BF16, 0, 5, 5, 32, 3, 3, 1, 1, 1, 1, None, cci.BF16, None,
                               16, 8, 2, None, None, cci.BF16, None) == cci.OK


def test_conv_geometry_errors():
    args = dict(O=16, G=8, K=2)
    bad = [(1, 5, 5, 32, 3, 3, 0, 1, 1, 1),   # stride 0
           (1, 5, 5, 32, 3, 3, 1, 1, -1, 1),  # negative pad
           (1, 1, 1, 32, 3, 3, 1, 1, 0, 0),   # kernel larger than input
           (1, 5, 5, 0, 3, 3, 1, 1, 1, 1)]    # Cin 0
    for B, H, W, Cin, KH, KW, sh, sw, ph, pw in bad:
        assert lib.cci_conv_im2col(FAKE, cci.BF16, B, H, W, Cin, KH, KW, sh, sw, ph, pw, FAKE, cci.BF16,
                                   FAKE, args["O"], args["G"], args["K"], None, FAKE, cci.BF16,
                                   None) == cci.EINVAL


def test_auto_algo_cost_model():
    # bf16, tile-friendly: expanded MFMA work wins while K/G > 1/32; 3x3 convs over 32 / 64 channels into
    # 32 / 64 outputs keep the whole expanded tile in registers
    assert cci.auto_algo(torch.bfloat16, torch.bfloat16, 100352, 576, 64, 64, 8, 2) == "resident_mfma"
    assert cci.auto_algo(torch.bfloat16, torch.bfloat16, 100352, 288, 32, 32, 8, 2) == "resident_mfma"
    # k x k convolutions over a multiple of 64 channels into a multiple of 128 outputs: tap-chunk MFMA
    assert cci.auto_algo(torch.bfloat16, torch.bfloat16, 100352, 576, 64, 128, 8, 2) == "tap_tile_mfma"
    assert cci.auto_algo(torch.bfloat16, torch.bfloat16, 3136, 4608, 512, 512, 8, 2) == "tap_tile_mfma"
    assert cci.auto_algo(torch.bfloat16, torch.bfloat16, 4096, 4096, 4096, 512, 16, 1) == "tap_tile_mfma"
    # 64 outputs, or 64 input channels: the dense-tile kernels
    assert cci.auto_algo(torch.bfloat16, torch.bfloat16, 50000, 576, 64, 96, 16, 2) == "dense_tile_mfma"
    assert cci.auto_algo(torch.bfloat16, torch.bfloat16, 50000, 864, 96, 128, 8, 2) == "dense_tile_mfma"
    # large FC / 1x1 products (>= 128 tiles of 256 x 256): wide-tile MFMA, any K
    assert cci.auto_algo(torch.bfloat16, torch.bfloat16, 4096, 4096, 4096, 4096, 16, 1) == "wide_tile_mfma"
    assert cci.auto_algo(torch.bfloat16, torch.bfloat16, 4096, 4096, 4096, 4096, 64, 1) == "wide_tile_mfma"
    assert cci.auto_algo(torch.bfloat16, torch.bfloat16, 12544, 256, 256, 1024, 16, 4) == "wide_tile_mfma"
    # fewer tiles, or a reduction of 128 or less: the tap-chunk kernels (two 128 x 128 tiles per CU)
    assert cci.auto_algo(torch.bfloat16, torch.bfloat16, 50176, 128, 128, 512, 8, 2) == "tap_tile_mfma"
    assert cci.auto_algo(torch.bfloat16, torch.bfloat16, 12544, 1024, 1024, 256, 16, 4) == "tap_tile_mfma"
    assert cci.auto_algo(torch.bfloat16, torch.bfloat16, 6000, 1024, 1024, 256, 16, 4) == "tap_tile_mfma"
    # G the vector kernels do not support: the tile path even at K/G < 1/32
    assert cci.auto_algo(torch.bfloat16, torch.bfloat16, 4096, 4096, 4096, 512, 64, 1) == "dense_tile_mfma"
    # fp32, or a reduction the tile path cannot step through: sparse-MAC
    assert cci.auto_algo(torch.float32, torch.float32, 64, 256, 256, 256, 8, 4) == "sparse_mac"
    assert cci.auto_algo(torch.bfloat16, torch.bfloat16, 1000, 147, 3, 64, 8, 8) == "sparse_mac"
    assert cci.auto_algo(torch.bfloat16, torch.bfloat16, 1000, 45, 45, 64, 8, 2) == "sparse_mac"
    # short reductions the tile path cannot step through (MobileNetV2's 16 / 24 / 144 channels)
    assert cci.auto_algo(torch.bfloat16, torch.bfloat16, 802816, 16, 16, 96, 8, 2) == "narrow_mfma"
    assert cci.auto_algo(torch.bfloat16, torch.bfloat16, 200704, 144, 144, 24, 8, 1) == "narrow_mfma"
    # small-Cin convs read through implicit im2col (a stem padded to 4 channels and KW = 8)
    assert cci.auto_algo(torch.bfloat16, torch.bfloat16, 802816, 224, 4, 64, 8, 8) == "narrow_mfma"
    assert cci.auto_algo(torch.bfloat16, torch.bfloat16, 5000, 216, 24, 64, 8, 2) == "narrow_mfma"
    # large 1x1 products with C <= 128 too, unless the tap-chunk kernels take them (O % 128 == 0);
    # C = 256 or fewer rows stay on the tile kernels
    assert cci.auto_algo(torch.bfloat16, torch.bfloat16, 200704, 128, 128, 96, 8, 2) == "narrow_mfma"
    assert cci.auto_algo(torch.bfloat16, torch.bfloat16, 200704, 128, 128, 256, 8, 2) == "tap_tile_mfma"
    # one 64-channel chunk over >= 100 K rows: the streaming kernels
    assert cci.auto_algo(torch.bfloat16, torch.bfloat16, 200704, 64, 64, 256, 8, 2) == "stream_tile_mfma"
    assert cci.auto_algo(torch.bfloat16, torch.bfloat16, 200704, 64, 64, 64, 8, 2) == "stream_tile_mfma"
    assert cci.auto_algo(torch.bfloat16, torch.bfloat16, 50176, 64, 64, 256, 8, 2) == "dense_tile_mfma"
    assert cci.auto_algo(torch.bfloat16, torch.bfloat16, 200704, 256, 256, 64, 8, 2) == "dense_tile_mfma"
    assert cci.auto_algo(torch.bfloat16, torch.bfloat16, 12544, 64, 64, 384, 8, 2) == "dense_tile_mfma"
    assert cci.auto_algo(torch.bfloat16, torch.bfloat16, 12544, 64, 64, 96, 8, 2) == "dense_tile_mfma"
    # long reductions over few row tiles (MobileNetV2's late projections at batch 64): split-reduction
    # kernels when 64 x 32 tiles fill one round of the chip, else tap-chunk 64-output tiles (O % 64 == 0);
    # from 12 544 rows, and for O % 128 == 0, the routes above
    assert cci.auto_algo(torch.bfloat16, torch.bfloat16, 3136, 960, 960, 160, 8, 2) == "split_k_mfma"
    assert cci.auto_algo(torch.bfloat16, torch.bfloat16, 3136, 576, 576, 160, 8, 4) == "split_k_mfma"
    assert cci.auto_algo(torch.bfloat16, torch.bfloat16, 3136, 960, 960, 320, 8, 2) == "tap_tile_mfma"
    assert cci.auto_algo(torch.bfloat16, torch.bfloat16, 12544, 576, 576, 96, 8, 2) == "dense_tile_mfma"
    assert cci.auto_algo(torch.bfloat16, torch.bfloat16, 12544, 384, 384, 64, 8, 2) == "dense_tile_mfma"
    assert cci.auto_algo(torch.bfloat16, torch.bfloat16, 3136, 512, 512, 128, 8, 2) == "tap_tile_mfma"
    assert cci.auto_algo(torch.bfloat16, torch.bfloat16, 3136, 960, 960, 160, 8, 8) == "dense_tile_mfma"
    assert cci.auto_algo(torch.bfloat16, torch.bfloat16, 512, 512, 512, 320, 4, 1) == "split_k_mfma"
    assert cci.auto_algo(torch.bfloat16, torch.bfloat16, 4096, 512, 512, 96, 16, 4) == "dense_tile_mfma"


@pytest.mark.skipif(torch.cuda.is_available(), reason="checks the no-device error path only")
def test_launch_without_device_reports_hip_error():
    # passes validation, then the HIP runtime refuses: CCI_EHIP, message set
    st = lib.cci_pack(FAKE, 16, 8, 8, 2, FAKE, cci.F32, FAKE, None)
    assert st == cci.EHIP
    assert lib.cci_last_error()


def test_bbs_and_2of4_validation():
    vb, ib = ctypes.c_size_t(0), ctypes.c_size_t(0)
    assert lib.cci_bbs_packed_sizes(8, 64, 4, 2, cci.BF16, ctypes.byref(vb), ctypes.byref(ib)) == cci.OK
    assert (vb.value, ib.value) == (8 * 16 * 2 * 2, 8 * 16 * 2)
    # balanced groups run along C: C % G != 0 is invalid (O need not divide)
    assert lib.cci_bbs_packed_sizes(7, 62, 4, 2, cci.BF16, ctypes.byref(vb), ctypes.byref(ib)) == cci.EINVAL
    assert lib.cci_bbs_pack(FAKE, 7, 62, 4, 2, FAKE, cci.BF16, FAKE, None) == cci.EINVAL
    assert lib.cci_bbs_pack(FAKE_MIS, 7, 64, 4, 2, FAKE, cci.BF16, FAKE, None) == cci.EALIGN
    assert lib.cci_2of4_sizes(32, 128, ctypes.byref(vb), ctypes.byref(ib)) == cci.OK
    assert (vb.value, ib.value) == (32 * 128, 32 * 128 // 8)
    assert lib.cci_2of4_sizes(24, 128, ctypes.byref(vb), ctypes.byref(ib)) == cci.EUNSUPPORTED   # M % 16
    assert lib.cci_2of4_sizes(32, 96, ctypes.byref(vb), ctypes.byref(ib)) == cci.EUNSUPPORTED    # R % 64
    # more than 2 kept weights per run of 4, fp32 values, G not a multiple of 4
    assert lib.cci_bbs_to_2of4(FAKE, cci.BF16, FAKE, 32, 128, 8, 3, FAKE, FAKE, None) == cci.EUNSUPPORTED
    assert lib.cci_bbs_to_2of4(FAKE, cci.F32, FAKE, 32, 128, 4, 2, FAKE, FAKE, None) == cci.EUNSUPPORTED
    assert lib.cci_bbs_to_2of4(FAKE, cci.BF16, FAKE, 32, 120, 6, 1, FAKE, FAKE, None) == cci.EUNSUPPORTED
    assert lib.cci_to_2of4_transposed(FAKE, cci.BF16, FAKE, 128, 32, 16, 4, FAKE, FAKE, None) == cci.EUNSUPPORTED
    assert lib.cci_to_2of4_transposed(FAKE, cci.BF16, FAKE, 130, 32, 16, 2, FAKE, FAKE, None) == cci.EINVAL
    assert lib.cci_spmm_2of4(FAKE, cci.F32, 4, 64, FAKE, FAKE, 16, None, FAKE, cci.BF16, None) == cci.EUNSUPPORTED
    assert lib.cci_spmm_2of4(FAKE, cci.BF16, 4, 64, FAKE, FAKE, 20, None, FAKE, cci.BF16, None) == cci.EUNSUPPORTED
    assert lib.cci_spmm_2of4(FAKE, cci.BF16, -1, 64, FAKE, FAKE, 16, None, FAKE, cci.BF16, None) == cci.EINVAL
    assert lib.cci_spmm_2of4(None, cci.BF16, 0, 64, None, None, 16, None, None, cci.BF16, None) == cci.OK
    assert lib.cci_spmm_2of4(FAKE, cci.BF16, 4, 64, FAKE_MIS, FAKE, 16, None, FAKE, cci.BF16, None) == cci.EALIGN


def test_td_schedule_host_logic_matches_oracle():
    import oracle
    for total in (1, 7, 100, 1001):
        for G, K in ((8, 2), (16, 1), (4, 4), (256, 3)):
            for step in sorted({0, 1, total // 3, total // 2, total // 2 + 1, total - 1, total}):
                assert cci.td_schedule(step, total, G, K) == oracle.td_schedule(step, total, G, K)
    n, p = ctypes.c_int32(7), ctypes.c_double(7.0)
    assert lib.cci_td_schedule(5, 4, 8, 2, ctypes.byref(n), ctypes.byref(p)) == cci.EINVAL
    assert n.value == 7 and p.value == 7.0


def test_td_mask_and_grad_validation():
    assert lib.cci_td_mask(FAKE, 16, 8, 8, 9, FAKE, ctypes.c_double(0.5), FAKE, cci.BF16, FAKE, None) == cci.EINVAL
    assert lib.cci_td_mask(FAKE, 16, 8, 8, 2, FAKE, ctypes.c_double(1.5), FAKE, cci.BF16, FAKE, None) == cci.EINVAL
    assert lib.cci_td_mask(FAKE, 12, 8, 8, 2, FAKE, ctypes.c_double(0.5), FAKE, cci.BF16, FAKE, None) == cci.EINVAL
    assert lib.cci_td_mask(FAKE, 16, 8, 8, 2, FAKE_MIS, ctypes.c_double(0.5), FAKE, cci.BF16, FAKE, None) == cci.EALIGN
    assert lib.cci_grad_packed(FAKE, FAKE, cci.BF16, 4, 8, FAKE, 16, 8, 9, FAKE, None) == cci.EINVAL
    assert lib.cci_grad_packed(FAKE, FAKE, cci.BF16, -1, 8, FAKE, 16, 8, 2, FAKE, None) == cci.EINVAL
    assert lib.cci_grad_packed(FAKE, FAKE, cci.BF16, 4, 8, FAKE, 16, 8, 2, FAKE_MIS, None) == cci.EALIGN


def test_index_width_host_logic_and_bits_validation():
    import oracle
    for G in range(1, 257):
        assert cci.index_width(G) == oracle.index_width(G)
    assert lib.cci_index_width(0) == -1 and lib.cci_index_width(257) == -1
    nb = ctypes.c_size_t(0)
    assert lib.cci_index_stream_bytes(33, 3, ctypes.byref(nb)) == cci.OK and nb.value == 16
    assert lib.cci_index_stream_bytes(33, 9, ctypes.byref(nb)) == cci.EINVAL
    assert lib.cci_index_bits(FAKE, 10, 0, FAKE, None) == cci.EINVAL
    assert lib.cci_index_bits(FAKE_MIS, 10, 3, FAKE, None) == cci.EALIGN
    # too few bits for G, unsupported row count, fp32
    assert lib.cci_spmm_bits(FAKE, cci.BF16, 4, 64, FAKE, cci.BF16, FAKE, 3, 64, 16, 2, None, FAKE, cci.BF16,
                             None) == cci.EINVAL
    assert lib.cci_spmm_bits(FAKE, cci.BF16, 65, 64, FAKE, cci.BF16, FAKE, 4, 64, 16, 2, None, FAKE, cci.BF16,
                             None) == cci.EUNSUPPORTED
    assert lib.cci_spmm_bits(FAKE, cci.F32, 4, 64, FAKE, cci.F32, FAKE, 4, 64, 16, 2, None, FAKE, cci.F32,
                             None) == cci.EUNSUPPORTED
    assert lib.cci_spmm_bits(None, cci.BF16, 0, 64, None, cci.BF16, None, 4, 64, 16, 2, None, None, cci.BF16,
                             None) == cci.OK
