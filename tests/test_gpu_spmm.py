"""cci_spmm on the GPU vs the oracle (Alg. 1 in double), both kernel families."""
import numpy as np
import pytest
import torch

import oracle
from gpu_common import (DEV, Guarded, epilogue_terms, need_gpu, oracle_pack_vals, rand_epilogue, tol_for,
                        x_as_f32)
from parity import check_close, to_np_f32
from paper_1910_11971_amd import workloads

pytestmark = pytest.mark.gpu


def run_case(X: torch.Tensor, W: np.ndarray, G, K, y_dtype, algo, *, rows=None, ep=None, seed=0):
    from paper_1910_11971_amd import cci
    vdt = torch.float32 if X.dtype == torch.float32 else torch.bfloat16
    N, C = X.shape
    O = W.shape[0]
    s, b, r, r_t, relu = ep if ep is not None else (None, None, None, None, False)
    Xd = X.to(DEV)
    vals, idx = cci.pack(torch.from_numpy(W).to(DEV), G, K, vdt)
    kw = {}
    if s is not None:
        kw["scale"] = torch.from_numpy(s).to(DEV)
    if b is not None:
        kw["bias"] = torch.from_numpy(b).to(DEV)
    if r_t is not None:
        kw["residual"] = r_t.to(DEV)
    Yg = Guarded((N, O), y_dtype)
    Y = cci.spmm(Xd, vals, idx, G, relu=relu, out_dtype=y_dtype, algo=algo, out=Yg.t, **kw)
    torch.cuda.synchronize()
    Yg.check(f"spmm {algo} N={N} C={C} O={O} G={G} K={K}")
    v_ref, idx_ref, _ = oracle_pack_vals(W, G, K, vdt)
    Yref, Yabs = oracle.spmm_rows(x_as_f32(X), v_ref, idx_ref, G, scale=s, bias=b, residual=r,
                                  relu=relu, rows=rows, want_abs=True)
    got = to_np_f32(Y)
    if rows is not None:
        got = got[rows]
    S = epilogue_terms(Yabs, s, b, None if r is None else (r if rows is None else r[rows]))
    return check_close(got, Yref, S, tol_for(y_dtype, X.dtype), f"spmm {algo} N={N} C={C} O={O} G={G} K={K}")


def rand_x(N, C, dtype, seed):
    rng = np.random.default_rng(seed)
    return torch.from_numpy(rng.standard_normal((N, C)).astype(np.float32)).to(dtype)


def rand_w(O, C, seed):
    return (np.random.default_rng(seed + 1).standard_normal((O, C)) / np.sqrt(C)).astype(np.float32)


CASES = [  # N, C, O, G, K
    (1, 32, 64, 8, 2), (37, 64, 64, 8, 2), (300, 96, 128, 16, 4), (1000, 256, 192, 8, 3),
    (129, 32, 64, 2, 1), (70, 64, 64, 4, 4), (513, 128, 64, 32, 7), (2047, 64, 256, 16, 1),
    (4500, 160, 64, 8, 8), (64, 576, 64, 8, 2),
]


@pytest.mark.parametrize("algo", ["sparse_mac", "dense_tile_mfma"])
@pytest.mark.parametrize("N,C,O,G,K", CASES)
def test_spmm_bf16(N, C, O, G, K, algo):
    need_gpu()
    run_case(rand_x(N, C, torch.bfloat16, N + C), rand_w(O, C, O + G), G, K, torch.bfloat16, algo)


WIDE_CASES = [  # N, C, O, G, K: chunks 1..5, ragged pixel blocks, every unit count, K == G
    (600, 256, 512, 8, 2), (300, 128, 256, 16, 1), (257, 64, 256, 16, 4), (1000, 320, 256, 4, 3),
    (512, 192, 768, 16, 16), (100, 256, 256, 64, 7), (2065, 128, 256, 2, 1), (1024, 128, 1024, 8, 2),
    (2048, 64, 256, 32, 9), (520, 128, 256, 32, 2), (300, 192, 512, 64, 4),
    # >= 128 tiles of 256 pixels: the 256-pixel plan (the rest run 128-pixel tiles)
    (32768, 64, 256, 64, 7), (32768, 128, 256, 4, 3), (33000, 64, 256, 32, 2), (32768, 192, 256, 16, 16),
    # 9, 10, 15 and 16 chunks: the six-chunk steady state, the one-chunk loop and the tails
    (300, 576, 256, 16, 1), (520, 640, 256, 16, 2), (300, 1024, 512, 16, 4), (257, 960, 256, 8, 8),
    (600, 576, 256, 32, 3), (300, 1024, 256, 64, 7), (130, 960, 256, 16, 8), (32768, 576, 256, 16, 1),
]


@pytest.mark.parametrize("N,C,O,G,K", WIDE_CASES)
def test_spmm_bf16_wide_tile(N, C, O, G, K):
    need_gpu()
    run_case(rand_x(N, C, torch.bfloat16, N + C), rand_w(O, C, O + G), G, K, torch.bfloat16, "wide_tile_mfma")


NARROW_CASES = [  # N, C, O, G, K: every k-step count 1..8, ragged N and O, one to 30 slices, G 2..256
    (1, 8, 16, 8, 2), (37, 16, 96, 8, 2), (1000, 24, 144, 8, 3), (333, 40, 36, 4, 1),
    (2049, 72, 100, 4, 4), (129, 104, 64, 16, 5), (700, 136, 24, 8, 1), (90, 168, 192, 32, 7),
    (515, 200, 80, 16, 16), (300, 256, 960, 64, 9), (5000, 144, 32, 8, 2), (64, 32, 256, 256, 3),
    (4500, 64, 8, 2, 1),
    # waves that stream more than one pixel group
    (3000, 256, 960, 64, 9), (70000, 136, 24, 8, 1),
]


@pytest.mark.parametrize("N,C,O,G,K", NARROW_CASES)
def test_spmm_bf16_narrow(N, C, O, G, K):
    need_gpu()
    run_case(rand_x(N, C, torch.bfloat16, N + C), rand_w(O, C, O + G), G, K, torch.bfloat16, "narrow_mfma")


TAP_FC_CASES = [  # N, C, O, G, K: FC products on the tap-chunk kernels
    (1, 64, 128, 8, 2), (129, 128, 256, 16, 4), (300, 640, 128, 4, 1), (1000, 1024, 256, 16, 4),
    (257, 192, 384, 32, 5), (2049, 64, 128, 8, 8), (777, 320, 128, 2, 1), (12544, 256, 256, 8, 3),
    (300, 128, 128, 8, 4), (300, 128, 128, 32, 16),
    # >= 257 workgroups: two workgroups per CU (the rest: one per CU)
    (33024, 64, 128, 8, 2), (33024, 128, 128, 32, 5), (16500, 192, 256, 16, 16), (40000, 320, 128, 4, 2),
    # 64-output tiles: O % 128 != 0, or fewer than 256 tiles of 128 outputs
    (500, 256, 320, 8, 2), (40000, 128, 64, 8, 2), (3000, 512, 512, 16, 4), (777, 192, 192, 16, 16),
]


@pytest.mark.parametrize("N,C,O,G,K", TAP_FC_CASES)
def test_spmm_bf16_tap_tile(N, C, O, G, K):
    need_gpu()
    run_case(rand_x(N, C, torch.bfloat16, N + C), rand_w(O, C, O + G), G, K, torch.bfloat16, "tap_tile_mfma")


STREAM_FC_CASES = [  # N, C, O, G, K: FC products on the streaming kernels (C <= 256)
    (1, 64, 64, 8, 2), (127, 128, 128, 16, 4), (128, 64, 128, 8, 8), (129, 192, 256, 32, 5),
    (1000, 256, 320, 4, 1), (5000, 192, 192, 2, 2), (3000, 256, 128, 1, 1), (777, 128, 384, 32, 32),
    # many row tiles per workgroup, 128- and 64-output tiles, a ragged last tile
    (33001, 64, 256, 8, 2), (40000, 128, 512, 8, 2), (70001, 256, 64, 8, 2), (20000, 192, 128, 16, 3),
    # 64-output tiles holding two 32-row groups; a three-chunk reduction with a ragged last row tile
    (2000, 64, 192, 32, 7), (9999, 192, 320, 32, 32),
]


@pytest.mark.parametrize("N,C,O,G,K", STREAM_FC_CASES)
def test_spmm_bf16_stream_tile(N, C, O, G, K):
    need_gpu()
    run_case(rand_x(N, C, torch.bfloat16, N + C), rand_w(O, C, O + G), G, K, torch.bfloat16, "stream_tile_mfma")


@pytest.mark.parametrize("y_dtype", [torch.bfloat16, torch.float32])
def test_spmm_stream_tile_large_sampled(y_dtype):
    """ResNet-50 layer1-shaped product (200 704 rows, 64 -> 256) with every
    epilogue term: a row of every 128-row tile against the oracle, plus the
    first and last tiles whole."""
    need_gpu()
    N, C, O, G, K = 200704, 64, 256, 8, 2
    rng = np.random.default_rng(31)
    rows = np.unique(np.concatenate([np.arange(0, 128), np.arange(N - 128, N),
                                     np.arange(0, N, 128) + rng.integers(0, 128, N // 128)]))
    ep = rand_epilogue(O, N, y_dtype, 32, residual=True, relu=True)
    run_case(rand_x(N, C, torch.bfloat16, 33), rand_w(O, C, 34), G, K, y_dtype, "stream_tile_mfma", rows=rows, ep=ep)


@pytest.mark.parametrize("residual", [False, True])
def test_spmm_auto_single_chunk_large(residual):
    """AUTO's route for one 64-channel chunk over >= 100 K rows (the streaming
    kernels), with and without a residual."""
    need_gpu()
    from paper_1910_11971_amd import cci
    N, C, O, G, K = 100352, 64, 128, 8, 2
    assert cci.auto_algo(torch.bfloat16, torch.bfloat16, N, C, C, O, G, K) == "stream_tile_mfma"
    rows = np.unique(np.concatenate([np.arange(0, 256), np.arange(N - 200, N), np.arange(0, N, 61)]))
    ep = rand_epilogue(O, N, torch.bfloat16, 41, residual=residual, relu=True)
    run_case(rand_x(N, C, torch.bfloat16, 42), rand_w(O, C, 43), G, K, torch.bfloat16, "auto", rows=rows, ep=ep)


def test_spmm_stream_tile_refuses_unsupported():
    need_gpu()
    from paper_1910_11971_amd import cci
    for C, O, G in ((320, 128, 8), (96, 128, 8), (128, 96, 8), (128, 128, 64)):
        X = rand_x(300, C, torch.bfloat16, 1).to(DEV)
        vals, idx = cci.pack(torch.from_numpy(rand_w(O, C, 2)).to(DEV), G, 2, torch.bfloat16)
        with pytest.raises(cci.CCIError):
            cci.spmm(X, vals, idx, G, algo="stream_tile_mfma")


SPLIT_K_CASES = [  # N, C, O, G, K
    # one k-step (seven idle waves), fewer k-steps than waves, a 16-output tile
    (1, 32, 16, 8, 2), (37, 64, 48, 8, 2), (200, 160, 32, 2, 1),
    # 32 x 64 tiles; 64 x 32 tiles; 32 x 32 tiles (K = 4); 32 x 16 tiles; ragged last row tiles
    (9999, 384, 128, 8, 2), (20001, 576, 96, 8, 2), (3136, 960, 320, 8, 4), (3136, 960, 160, 8, 2),
    (5000, 256, 64, 16, 3), (12544, 512, 64, 32, 1), (3000, 256, 128, 1, 1),
    # groups straddling 16-output tiles (G = 12), a group wider than the tile (G = 64), K == G
    (700, 192, 96, 12, 3), (500, 256, 128, 64, 2), (1000, 96, 64, 4, 4),
    # a reduction of 16 k-steps per wave: four load batches
    (100, 4096, 64, 16, 4),
]


@pytest.mark.parametrize("N,C,O,G,K", SPLIT_K_CASES)
def test_spmm_bf16_split_k(N, C, O, G, K):
    need_gpu()
    run_case(rand_x(N, C, torch.bfloat16, N + C), rand_w(O, C, O + G), G, K, torch.bfloat16, "split_k_mfma")


# Packed rows of a tile's groups too large for LDS beside the partial tiles
# (many small groups over a long reduction): every lane loads its own group's
# entries per k-step.  32 x 16, 32 x 32, 64 x 32 and 128 x 32 tiles, with
# 2 to 6 load batches per wave.
SPLIT_K_DIRECT_CASES = [(300, 3264, 16, 2, 2), (2000, 2048, 64, 2, 2), (5000, 1344, 64, 2, 2),
                        (5000, 1344, 128, 4, 4)]


@pytest.mark.parametrize("N,C,O,G,K", SPLIT_K_DIRECT_CASES)
def test_spmm_bf16_split_k_direct_loads(N, C, O, G, K):
    need_gpu()
    run_case(rand_x(N, C, torch.bfloat16, N + C), rand_w(O, C, O + G), G, K, torch.bfloat16, "split_k_mfma")


@pytest.mark.parametrize("N,C,O", [(3136, 960, 160), (3136, 960, 320), (3136, 576, 160), (12544, 576, 96),
                                   (12544, 384, 64)])
@pytest.mark.parametrize("y_dtype", [torch.bfloat16, torch.float32])
def test_spmm_split_k_mobilenetv2_projections(N, C, O, y_dtype):
    """MobileNetV2's late projecting 1x1 layers at batch 64 (G = 8, K = 2)
    with batch norm folded into scale / bias and a residual: every output."""
    need_gpu()
    ep = rand_epilogue(O, N, y_dtype, N + O, residual=True, relu=False)
    run_case(rand_x(N, C, torch.bfloat16, C), rand_w(O, C, O), 8, 2, y_dtype, "split_k_mfma", ep=ep)


def test_spmm_split_k_refuses_unsupported():
    need_gpu()
    from paper_1910_11971_amd import cci
    for C, O, G, K in ((48, 64, 8, 2), (960, 24, 8, 2), (960, 160, 8, 5)):
        X = rand_x(300, C, torch.bfloat16, 1).to(DEV)
        vals, idx = cci.pack(torch.from_numpy(rand_w(O, C, 2)).to(DEV), G, K, torch.bfloat16)
        with pytest.raises(cci.CCIError):
            cci.spmm(X, vals, idx, G, algo="split_k_mfma")


def test_spmm_wide_tile_repeat_is_identical():
    """Two launches on the same inputs give the same bytes (no state carried between launches)."""
    need_gpu()
    from paper_1910_11971_amd import cci
    X = rand_x(700, 256, torch.bfloat16, 3).to(DEV)
    vals, idx = cci.pack(torch.from_numpy(rand_w(512, 256, 4)).to(DEV), 8, 2, torch.bfloat16)
    Y1 = cci.spmm(X, vals, idx, 8, algo="wide_tile_mfma")
    Y2 = cci.spmm(X, vals, idx, 8, algo="wide_tile_mfma")
    torch.cuda.synchronize()
    assert torch.equal(Y1.view(torch.int16), Y2.view(torch.int16))


@pytest.mark.parametrize("algo", ["sparse_mac", "dense_tile_mfma", "wide_tile_mfma", "narrow_mfma", "tap_tile_mfma",
                                  "stream_tile_mfma", "split_k_mfma"])
def test_spmm_bf16_in_f32_out_with_epilogue(algo):
    need_gpu()
    N, C, O, G, K = 777, 128, 256, 8, 2
    ep = rand_epilogue(O, N, torch.float32, 3, residual=True, relu=True)
    run_case(rand_x(N, C, torch.bfloat16, 1), rand_w(O, C, 2), G, K, torch.float32, algo, ep=ep)


@pytest.mark.parametrize("algo", ["sparse_mac", "dense_tile_mfma", "wide_tile_mfma", "narrow_mfma", "tap_tile_mfma",
                                  "stream_tile_mfma", "split_k_mfma"])
def test_spmm_bf16_epilogue_bf16_residual(algo):
    need_gpu()
    N, C, O, G, K = 300, 64, 256, 16, 4
    ep = rand_epilogue(O, N, torch.bfloat16, 4, residual=True, relu=True)
    run_case(rand_x(N, C, torch.bfloat16, 5), rand_w(O, C, 6), G, K, torch.bfloat16, algo, ep=ep)


@pytest.mark.parametrize("N,C,O,G,K", [(64, 256, 256, 8, 4), (5, 33, 16, 4, 2), (300, 45, 96, 32, 3),
                                       (1000, 7, 8, 2, 1)])
def test_spmm_fp32(N, C, O, G, K):
    need_gpu()
    run_case(rand_x(N, C, torch.float32, N), rand_w(O, C, C), G, K, torch.float32, "auto")


FEW_ROW_CASES = [  # N, C, O, G, K: N <= 64 bf16 products (the library's choice: the few-row kernel)
    (1, 64, 16, 8, 2), (17, 96, 48, 16, 4), (64, 512, 256, 8, 3), (33, 32, 48, 3, 2), (5, 256, 256, 256, 9),
    (64, 160, 64, 4, 4), (2, 1024, 512, 64, 1),
]


@pytest.mark.parametrize("N,C,O,G,K", FEW_ROW_CASES)
def test_spmm_bf16_few_rows(N, C, O, G, K):
    need_gpu()
    from paper_1910_11971_amd import cci
    assert cci.auto_algo(torch.bfloat16, torch.bfloat16, N, C, C, O, G, K) == "few_rows_mfma"
    run_case(rand_x(N, C, torch.bfloat16, N + C + 1), rand_w(O, C, O + G + 1), G, K, torch.bfloat16, "auto")
    run_case(rand_x(N, C, torch.bfloat16, N + C + 2), rand_w(O, C, O + G + 2), G, K, torch.bfloat16, "few_rows_mfma")


@pytest.mark.parametrize("N,C,O,G,K", [(64, 2048, 1000, 8, 8), (17, 96, 52, 4, 2), (33, 128, 36, 4, 4),
                                       (7, 64, 24, 8, 3)])
def test_spmm_bf16_few_rows_ragged_tile(N, C, O, G, K):
    """O % 16 != 0 (a last tile of 4, 8 or 12 outputs) on the pinned few-row kernel."""
    need_gpu()
    run_case(rand_x(N, C, torch.bfloat16, N + C + 3), rand_w(O, C, O + G + 3), G, K, torch.bfloat16, "few_rows_mfma")


@pytest.mark.parametrize("O", [128, 1000])
@pytest.mark.parametrize("y_dtype", [torch.bfloat16, torch.float32])
def test_spmm_few_rows_epilogue(y_dtype, O):
    need_gpu()
    N, C, G, K = 40, 256, 8, 2
    ep = rand_epilogue(O, N, y_dtype, 23, residual=True, relu=True)
    run_case(rand_x(N, C, torch.bfloat16, 24), rand_w(O, C, 25), G, K, y_dtype, "few_rows_mfma", ep=ep)


def test_spmm_odd_c_bf16_auto_routes_to_sparse_mac():
    need_gpu()
    run_case(rand_x(200, 45, torch.bfloat16, 9), rand_w(32, 45, 9), 8, 2, torch.bfloat16, "auto")


def test_spmm_fc256_full():
    """Single FC layer, fp32, X [64,256], W [256,256], G=8, K=4 -- every output."""
    need_gpu()
    wl = workloads.WORKLOADS["fc256"]
    X, W = workloads.draw(wl)
    run_case(X, W, wl.G, wl.K, torch.float32, "auto")


@pytest.mark.parametrize("xdt", [torch.bfloat16, torch.float32])
@pytest.mark.parametrize("N,C,O,G,K", [(200, 96, 128, 16, 4), (64, 256, 256, 32, 7), (256, 40, 64, 16, 16),
                                       (3, 520, 96, 32, 1)])
def test_spmm_sparse_mac_small_n_wide_groups(N, C, O, G, K, xdt):
    """Products with at most 256 rows take the wave-per-(row, group) variant
    of the vector kernels: G = 16 and 32 (the 64-lane reduction and the
    lane < G store select), with every epilogue term."""
    need_gpu()
    ep = rand_epilogue(O, N, xdt, 17, residual=True, relu=True)
    run_case(rand_x(N, C, xdt, N + 3), rand_w(O, C, O + 5), G, K, xdt, "sparse_mac", ep=ep)
