"""Pins for the CPU oracle: each check compares it with something other than
itself -- a value the paper fixes, a closed form, a brute force, or a library
routine -- so that a dropped term, wrong sign, wrong index or transposed
operand in the oracle fails at least one of them."""
import itertools
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle
from conftest import read_golden


def bf16_exact(x):
    return oracle.bf16_bits_to_f32(oracle.bf16_rne(x))


# ---------------------------------------------------------------- pack -----

def brute_force_keep(col, K):
    """All C(G,K) subsets; keep the one with the largest sum |w|; among equal
    sums the lexicographically smallest index tuple (ties -> lower rows)."""
    G = len(col)
    best, best_key = None, None
    for sub in itertools.combinations(range(G), K):
        s = sum(abs(float(col[r])) for r in sub)
        key = (s, tuple(-r for r in sub))
        if best_key is None or key > best_key:
            best, best_key = sub, key
    return best


@pytest.mark.parametrize("G,K", [(2, 1), (4, 1), (4, 2), (4, 3), (8, 2), (8, 5), (6, 4), (3, 2)])
def test_pack_matches_brute_force(G, K):
    rng = np.random.default_rng(G * 100 + K)
    O, C = 3 * G, 17
    W = rng.standard_normal((O, C)).astype(np.float32)
    vals, idx = oracle.pack(W, G, K)
    for g in range(O // G):
        for c in range(C):
            col = W[g * G:(g + 1) * G, c]
            keep = brute_force_keep(col, K)
            assert tuple(idx[g, :, c]) == keep
            np.testing.assert_array_equal(vals[g, :, c], col[list(keep)])


def test_pack_ties_go_to_lower_row():
    # equal magnitudes, mixed signs and signed zeros: lower r must win
    W = np.array([[1.0, 0.0, 2.0],
                  [-1.0, -0.0, 2.0],
                  [1.0, 0.0, -2.0],
                  [0.5, 0.0, 2.0]], np.float32)
    vals, idx = oracle.pack(W, 4, 2)
    assert idx[0, :, 0].tolist() == [0, 1]
    assert idx[0, :, 1].tolist() == [0, 1]
    assert idx[0, :, 2].tolist() == [0, 1]
    for c in range(3):
        assert brute_force_keep(W[:, c], 2) == tuple(idx[0, :, c])


def test_pack_invariants_and_sparsity():
    rng = np.random.default_rng(7)
    for G, K in [(8, 2), (16, 4), (16, 1), (4, 3)]:
        O, C = 4 * G, 33
        W = rng.standard_normal((O, C)).astype(np.float32)
        vals, idx = oracle.pack(W, G, K)
        assert vals.shape == idx.shape == (O // G, K, C)
        # strictly ascending indices in [0, G)
        assert (idx < G).all()
        if K > 1:
            assert (np.diff(idx.astype(int), axis=1) > 0).all()
        Wd = oracle.unpack(vals, idx, G)
        nnz = int((Wd != 0).sum())
        assert nnz == O * C * K // G                   # exactly K per group
        assert abs(1 - nnz / (O * C) - (1 - K / G)) < 1e-12   # sparsity 1 - K/G
        # every kept |w| >= every dropped |w| in its group
        for g in range(O // G):
            blk = np.abs(W[g * G:(g + 1) * G])
            kept = np.abs(Wd[g * G:(g + 1) * G]) > 0
            for c in range(C):
                assert blk[kept[:, c], c].min() >= blk[~kept[:, c], c].max() if K < G else True
        # kept values are exact copies
        np.testing.assert_array_equal(Wd[Wd != 0], W[Wd != 0])


def test_pack_special_cases():
    rng = np.random.default_rng(3)
    W = rng.standard_normal((16, 9)).astype(np.float32)
    # K = G: identity (dense control)
    np.testing.assert_array_equal(oracle.unpack(*oracle.pack(W, 8, 8), 8), W)
    # K = 1: argmax |w| per group column
    vals, idx = oracle.pack(W, 8, 1)
    for g in range(2):
        am = np.argmax(np.abs(W[g * 8:(g + 1) * 8]), axis=0)
        np.testing.assert_array_equal(idx[g, 0], am)
        np.testing.assert_array_equal(vals[g, 0], W[g * 8 + am, np.arange(9)])


def test_pack_column_permutation_invariance_and_row_equivariance():
    rng = np.random.default_rng(11)
    W = rng.standard_normal((24, 13)).astype(np.float32)
    G, K = 8, 3
    Wd = oracle.unpack(*oracle.pack(W, G, K), G)
    perm = rng.permutation(13)
    Wd_p = oracle.unpack(*oracle.pack(W[:, perm], G, K), G)
    np.testing.assert_array_equal(Wd_p, Wd[:, perm])
    rp = np.concatenate([g * G + rng.permutation(G) for g in range(3)])
    Wd_r = oracle.unpack(*oracle.pack(W[rp], G, K), G)
    np.testing.assert_array_equal(Wd_r, Wd[rp])


def test_pack_sec33_worked_example(golden_dir):
    d = read_golden(os.path.join(golden_dir, "sec33_worked_example.txt"))
    G, K = int(d["G"][0][0]), int(d["K"][0][0])
    W = np.array([float(v) for v in d["W"][0]], np.float32).reshape(G, 1)
    vals, idx = oracle.pack(W, G, K)
    assert int(idx[0, 0, 0]) == int(d["idx"][0][0])
    assert float(vals[0, 0, 0]) == float(d["val"][0][0])
    X = np.array([[float(d["x"][0][0])]], np.float32)
    Y = oracle.spmm_rows(X, vals, idx, G)
    np.testing.assert_array_equal(Y[0], np.array([float(v) for v in d["H"][0]]))


def test_fig1_hand_example(golden_dir):
    d = read_golden(os.path.join(golden_dir, "fig1_hand_example.txt"))
    G, K = int(d["G"][0][0]), int(d["K"][0][0])
    W = np.array(d["W"], dtype=np.float32)
    M = np.array(d["M"], dtype=np.float32)
    assert W.shape == (8, 5) and G == 4 and K == 2            # Fig. 1 shape
    vals, idx = oracle.pack(W, G, K)
    np.testing.assert_array_equal(idx.reshape(-1, 5), np.array(d["idx"], dtype=np.uint8))
    np.testing.assert_array_equal(vals.reshape(-1, 5), np.array(d["val"], dtype=np.float32))
    Wd = oracle.unpack(vals, idx, G)
    np.testing.assert_array_equal(Wd, M)
    assert int((Wd != 0).sum()) == 20 and (Wd == 0).mean() == 0.5   # 50% sparse
    X = np.array(d["X"], dtype=np.float32)
    Y = oracle.spmm_rows(X, vals, idx, G)
    np.testing.assert_array_equal(Y, np.array(d["Y"], dtype=np.float64))


def test_eq1_closed_form_values(golden_dir):
    with open(os.path.join(golden_dir, "eq1_values.txt")) as f:
        rows = [l.split() for l in f if l.strip() and not l.startswith("#")]
    for G, Ps, Pd in rows:
        assert oracle.eq1_pd(int(G), Fraction(Ps)) == Fraction(Pd)


def test_eq1_trends():
    # P_d rises as G falls (same Ps) and as Ps rises (same G)  (Sec. 4)
    for Ps in (Fraction(1, 2), Fraction(3, 4)):
        vals = [oracle.eq1_pd(G, Ps) for G in (4, 8, 16, 32, 64)]
        assert all(a > b for a, b in zip(vals, vals[1:]))
    assert oracle.eq1_pd(16, Fraction(1, 2)) < oracle.eq1_pd(16, Fraction(3, 4)) < \
        oracle.eq1_pd(16, Fraction(7, 8)) < oracle.eq1_pd(16, Fraction(15, 16))


@pytest.mark.parametrize("G,Ps", [(4, Fraction(1, 2)), (8, Fraction(3, 4)), (16, Fraction(3, 4))])
def test_pack_discard_rate_matches_eq1(G, Ps):
    """Monte-Carlo: i.i.d. weights, each zero w.p. Ps; the packer (K = s
    slots) must discard nonzeros at the rate Eq. 1 predicts."""
    s = int(G * (1 - Ps))
    rng = np.random.default_rng(G)
    O, C = G * 400, 2500                  # 10^6 groups
    W = rng.standard_normal((O, C)).astype(np.float32)
    W[rng.random((O, C)) < float(Ps)] = 0.0
    vals, idx = oracle.pack(W, G, s)
    nonzero = int((W != 0).sum())
    kept_nonzero = int((vals != 0).sum())
    est = (nonzero - kept_nonzero) / nonzero
    pd = float(oracle.eq1_pd(G, Ps))
    # binomial standard error over ~10^6 groups is < 5e-4; allow 6 sigma
    assert abs(est - pd) < 3e-3, (est, pd)


# ---------------------------------------------------------------- spmm -----

@pytest.mark.parametrize("G,K", [(8, 4), (8, 2), (16, 1), (4, 3), (2, 2)])
def test_spmm_equals_library_matmul_of_masked(G, K):
    rng = np.random.default_rng(G * 7 + K)
    N, C, O = 37, 45, 5 * G
    X = rng.standard_normal((N, C)).astype(np.float32)
    W = rng.standard_normal((O, C)).astype(np.float32)
    vals, idx = oracle.pack(W, G, K)
    Wd = oracle.unpack(vals, idx, G)
    Y = oracle.spmm_rows(X, vals, idx, G)
    ref = X.astype(np.float64) @ Wd.astype(np.float64).T        # numpy BLAS, float64
    np.testing.assert_allclose(Y, ref, rtol=1e-12, atol=1e-12)
    # Alg. 0 on the unpacked matrix: same terms in the same order
    Yd = oracle.dense_rows(X, Wd)
    assert np.array_equal(Y, Yd)
    # row subset gives the same rows
    rows = np.array([36, 0, 5, 5, 17])
    np.testing.assert_array_equal(oracle.spmm_rows(X, vals, idx, G, rows=rows), Y[rows])


def test_spmm_k_equals_g_is_plain_product():
    rng = np.random.default_rng(5)
    X = rng.standard_normal((9, 21)).astype(np.float32)
    W = rng.standard_normal((16, 21)).astype(np.float32)
    vals, idx = oracle.pack(W, 8, 8)
    np.testing.assert_allclose(oracle.spmm_rows(X, vals, idx, 8),
                               X.astype(np.float64) @ W.astype(np.float64).T, rtol=1e-12, atol=1e-12)


def test_spmm_single_nonzero_lands_on_group_row():
    # one-hot X column and one kept weight -> exactly val at row g*G + idx (Alg. 1)
    G, K, C = 8, 1, 6
    W = np.zeros((3 * G, C), np.float32)
    W[2 * G + 5, 4] = 1.75            # group 2, row 5, column 4
    vals, idx = oracle.pack(W, G, K)
    assert idx[2, 0, 4] == 5 and vals[2, 0, 4] == 1.75
    X = np.zeros((2, C), np.float32)
    X[1, 4] = 1.0
    Y = oracle.spmm_rows(X, vals, idx, G)
    expect = np.zeros((2, 3 * G))
    expect[1, 2 * G + 5] = 1.75
    np.testing.assert_array_equal(Y, expect)


def test_spmm_epilogue_terms():
    rng = np.random.default_rng(9)
    N, C, G, K = 6, 10, 4, 2
    O = 3 * G
    X = rng.standard_normal((N, C)).astype(np.float32)
    W = rng.standard_normal((O, C)).astype(np.float32)
    scale = rng.random(O).astype(np.float32) + 0.5
    bias = rng.standard_normal(O).astype(np.float32)
    res = rng.standard_normal((N, O)).astype(np.float32)
    vals, idx = oracle.pack(W, G, K)
    Wd = oracle.unpack(vals, idx, G).astype(np.float64)
    acc = X.astype(np.float64) @ Wd.T
    ref = np.maximum(acc * scale + bias + res, 0.0)
    Y = oracle.spmm_rows(X, vals, idx, G, scale=scale, bias=bias, residual=res, relu=True)
    np.testing.assert_allclose(Y, ref, rtol=1e-12, atol=1e-12)
    Y2, Yabs = oracle.spmm_rows(X, vals, idx, G, want_abs=True)
    np.testing.assert_allclose(Yabs, np.abs(X.astype(np.float64)) @ np.abs(Wd).T, rtol=1e-12)


# ---------------------------------------------------------------- conv -----

@pytest.mark.parametrize("k,stride,pad", [(3, 1, 1), (3, 2, 1), (1, 1, 0), (1, 2, 0), (7, 2, 3), (2, 1, 0)])
def test_conv_direct_matches_torch_conv2d(k, stride, pad):
    rng = np.random.default_rng(k * 10 + stride + pad)
    B, H, W, Cin, O = 2, 9, 11, 5, 8
    X = rng.standard_normal((B, H, W, Cin)).astype(np.float32)
    Wt = rng.standard_normal((O, k, k, Cin)).astype(np.float32)
    Y = oracle.conv2d_nhwc(X, Wt, (stride, stride), (pad, pad))
    ref = torch.nn.functional.conv2d(
        torch.from_numpy(X).double().permute(0, 3, 1, 2),
        torch.from_numpy(Wt).double().permute(0, 3, 1, 2), stride=stride, padding=pad)
    ref = ref.permute(0, 2, 3, 1).reshape(-1, O).numpy()
    np.testing.assert_allclose(Y, ref, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("k,stride,pad", [(3, 1, 1), (3, 2, 1), (1, 1, 0), (7, 2, 3), (2, 1, 0)])
def test_conv_abs_sum_matches_torch_conv2d_of_magnitudes(k, stride, pad):
    """Yabs (the per-output sum of |terms| that scales the GPU tolerance) is
    the convolution of |X| with |W|, zero padding included; it must not move
    with the epilogue, and a pixel subset must give the same rows."""
    rng = np.random.default_rng(100 + k * 10 + stride + pad)
    B, H, W, Cin, O = 2, 9, 11, 5, 8
    X = rng.standard_normal((B, H, W, Cin)).astype(np.float32)
    Wt = rng.standard_normal((O, k, k, Cin)).astype(np.float32)
    Wt[rng.random(Wt.shape) < 0.5] = 0.0  # masked weights contribute nothing
    sc = (0.5 + rng.random(O)).astype(np.float32)
    bi = rng.standard_normal(O).astype(np.float32)
    _, Yabs = oracle.conv2d_nhwc(X, Wt, (stride, stride), (pad, pad), scale=sc, bias=bi, relu=True,
                                 want_abs=True)
    ref = torch.nn.functional.conv2d(
        torch.from_numpy(np.abs(X)).double().permute(0, 3, 1, 2),
        torch.from_numpy(np.abs(Wt)).double().permute(0, 3, 1, 2), stride=stride, padding=pad)
    ref = ref.permute(0, 2, 3, 1).reshape(-1, O).numpy()
    np.testing.assert_allclose(Yabs, ref, rtol=1e-12, atol=1e-12)
    pix = np.array([0, 3, ref.shape[0] - 1], np.int64)
    _, Ysub = oracle.conv2d_nhwc(X, Wt, (stride, stride), (pad, pad), pixels=pix, want_abs=True)
    np.testing.assert_allclose(Ysub, ref[pix], rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("k,stride,pad", [(3, 1, 1), (3, 2, 1), (1, 2, 0)])
def test_im2col_matches_torch_unfold(k, stride, pad):
    rng = np.random.default_rng(1)
    B, H, W, Cin = 2, 7, 6, 3
    X = rng.standard_normal((B, H, W, Cin)).astype(np.float32)
    A = oracle.im2col_nhwc(X, k, k, (stride, stride), (pad, pad))
    U = torch.nn.functional.unfold(torch.from_numpy(X).double().permute(0, 3, 1, 2),
                                   kernel_size=k, stride=stride, padding=pad)   # [B, Cin*k*k, L]
    Ho, Wo = oracle.conv_out_hw(H, W, k, k, (stride, stride), (pad, pad))
    U = U.reshape(B, Cin, k, k, Ho * Wo).permute(0, 4, 2, 3, 1).reshape(B * Ho * Wo, k * k * Cin)
    np.testing.assert_array_equal(A, U.numpy().astype(np.float32))


def test_cci_conv_equals_im2col_then_alg1_and_1x1_equals_fc():
    rng = np.random.default_rng(21)
    B, H, W, Cin, O, G, K = 2, 8, 7, 6, 16, 8, 2
    X = rng.standard_normal((B, H, W, Cin)).astype(np.float32)
    Wm = rng.standard_normal((O, 3 * 3 * Cin)).astype(np.float32)
    vals, idx = oracle.pack(Wm, G, K)
    Wd = oracle.unpack(vals, idx, G).reshape(O, 3, 3, Cin)
    Yc = oracle.conv2d_nhwc(X, Wd, (1, 1), (1, 1))
    A = oracle.im2col_nhwc(X, 3, 3, (1, 1), (1, 1))
    Ys = oracle.spmm_rows(A, vals, idx, G)
    np.testing.assert_allclose(Yc, Ys, rtol=1e-12, atol=1e-12)
    # 1x1 stride-1 conv == FC on the flattened pixels
    W1 = rng.standard_normal((O, Cin)).astype(np.float32)
    v1, i1 = oracle.pack(W1, G, K)
    Y1 = oracle.conv2d_nhwc(X, oracle.unpack(v1, i1, G).reshape(O, 1, 1, Cin))
    Yf = oracle.spmm_rows(X.reshape(-1, Cin), v1, i1, G)
    np.testing.assert_allclose(Y1, Yf, rtol=1e-12, atol=1e-12)
    # pack is column-local: the mask does not depend on the column order
    perm = rng.permutation(9 * Cin)
    Wd_p = oracle.unpack(*oracle.pack(Wm[:, perm], G, K), G)
    np.testing.assert_array_equal(Wd_p, Wd.reshape(O, -1)[:, perm])


# ------------------------------------------------------------- rounding ----

def test_bf16_rne_matches_torch():
    rng = np.random.default_rng(0)
    x = np.concatenate([
        rng.standard_normal(100000).astype(np.float32),
        (rng.standard_normal(1000) * 1e30).astype(np.float32),
        (rng.standard_normal(1000) * 1e-38).astype(np.float32),
        np.array([0.0, -0.0, np.inf, -np.inf, 3.4e38, -3.4e38, 1e-45], np.float32),
    ])
    # exact ties: low 16 bits == 0x8000 with both parities of bit 16
    ties = (np.arange(2000, dtype=np.uint32) << 16 | 0x3f800000 | 0x8000).view(np.float32)
    x = np.concatenate([x, ties, -ties])
    got = oracle.bf16_rne(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(got, ref)
    # hand cases: 1 + 2^-8 (tie, even stays 1.0); 1 + 3*2^-8 (tie, odd rounds up)
    assert oracle.bf16_rne(np.array([1 + 2 ** -8], np.float32))[0] == 0x3F80
    assert oracle.bf16_rne(np.array([1 + 3 * 2 ** -8], np.float32))[0] == 0x3F82
    nan = oracle.bf16_rne(np.array([np.nan], np.float32))[0]
    assert (nan & 0x7F80) == 0x7F80 and (nan & 0x7F) != 0


# ---------------------------------------------------------------- glue -----

def test_maxpool_and_avgpool_match_library():
    rng = np.random.default_rng(4)
    X = rng.standard_normal((2, 9, 10, 3)).astype(np.float32)
    Y = oracle.maxpool2d_nhwc(X, 3, 2, 1)
    ref = torch.nn.functional.max_pool2d(torch.from_numpy(X).permute(0, 3, 1, 2), 3, 2, 1)
    np.testing.assert_array_equal(Y, ref.permute(0, 2, 3, 1).numpy())
    A = oracle.global_avgpool_nhwc(X)
    np.testing.assert_allclose(A, X.astype(np.float64).mean(axis=(1, 2)), rtol=1e-13)


def test_oracle_rejects_bad_arguments():
    W = np.zeros((12, 3), np.float32)
    with pytest.raises(ValueError):
        oracle.pack(W, 8, 2)          # O % G != 0
    with pytest.raises(ValueError):
        oracle.pack(W, 4, 5)          # K > G
    with pytest.raises(ValueError):
        oracle.pack(W, 4, 0)          # K < 1
