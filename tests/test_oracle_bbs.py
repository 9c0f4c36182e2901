"""Pins for the oracle's balanced-sparsity functions (Sec. 2.4, Sec. 3.3,
Fig. 2b): each compares it with something other than itself -- a brute force
over all subsets, the transpose relation to the CCI projection, a library
matmul, the dense triple loop, hand examples with exact small integers."""
import numpy as np
import pytest

import oracle
from test_oracle import brute_force_keep


@pytest.mark.parametrize("G,K", [(2, 1), (4, 1), (4, 2), (4, 3), (8, 2), (8, 5), (6, 4), (3, 2)])
def test_bbs_pack_matches_brute_force(G, K):
    rng = np.random.default_rng(G * 31 + K)
    O, C = 5, 4 * G
    W = rng.standard_normal((O, C)).astype(np.float32)
    vals, idx = oracle.bbs_pack(W, G, K)
    assert vals.shape == idx.shape == (O, C // G, K)
    for o in range(O):
        for j in range(C // G):
            grp = W[o, j * G:(j + 1) * G]
            keep = brute_force_keep(grp, K)
            assert tuple(idx[o, j]) == keep
            np.testing.assert_array_equal(vals[o, j], grp[list(keep)])


def test_bbs_pack_ties_go_to_lower_position():
    W = np.array([[1.0, -1.0, 1.0, 0.5, 0.0, -0.0, 0.0, 0.0]], np.float32)
    vals, idx = oracle.bbs_pack(W, 4, 2)
    assert idx[0].tolist() == [[0, 1], [0, 1]]
    assert vals[0, 0].tolist() == [1.0, -1.0]


@pytest.mark.parametrize("G,K", [(4, 2), (8, 3), (16, 1), (16, 16), (5, 2)])
def test_bbs_is_cci_of_the_transpose(G, K):
    """Balanced groups are G contiguous weights of one row; CCI groups are G
    contiguous weights of one column (Sec. 2.4, Fig. 2a vs 2b).  So the
    balanced projection of W is the CCI projection of W^T, slot for slot."""
    rng = np.random.default_rng(G + 7 * K)
    O, C = 24, 4 * G
    W = rng.standard_normal((O, C)).astype(np.float32)
    bv, bi = oracle.bbs_pack(W, G, K)                 # [O][C/G][K]
    cv, ci = oracle.pack(np.ascontiguousarray(W.T), G, K)  # [C/G][K][O]
    np.testing.assert_array_equal(bv, cv.transpose(2, 0, 1))
    np.testing.assert_array_equal(bi, ci.transpose(2, 0, 1))
    np.testing.assert_array_equal(oracle.bbs_unpack(bv, bi, G), oracle.unpack(cv, ci, G).T)


def test_bbs_pack_invariants_and_special_cases():
    rng = np.random.default_rng(3)
    O, C, G, K = 16, 64, 8, 3
    W = rng.standard_normal((O, C)).astype(np.float32)
    vals, idx = oracle.bbs_pack(W, G, K)
    assert (np.diff(idx.astype(int), axis=2) > 0).all() and idx.max() < G
    Wd = oracle.bbs_unpack(vals, idx, G)
    nz = (Wd != 0).reshape(O, C // G, G).sum(axis=2)
    assert (nz == K).all()                                   # exactly K kept per group
    assert np.count_nonzero(Wd) / Wd.size == pytest.approx(1 - (1 - K / G))
    mag = np.abs(W).reshape(O, C // G, G)
    kept = (Wd != 0).reshape(O, C // G, G)
    assert (np.where(kept, mag, np.inf).min(axis=2) >= np.where(kept, -np.inf, mag).max(axis=2)).all()
    # K = G keeps everything in place; K = 1 keeps each group's argmax |w|
    v, i = oracle.bbs_pack(W, G, G)
    np.testing.assert_array_equal(oracle.bbs_unpack(v, i, G), W)
    v, i = oracle.bbs_pack(W, G, 1)
    np.testing.assert_array_equal(i[:, :, 0], mag.argmax(axis=2))


def test_bbs_rejects_ragged_groups():
    with pytest.raises(ValueError):
        oracle.bbs_pack(np.ones((4, 10), np.float32), 4, 2)


@pytest.mark.parametrize("G,K", [(4, 2), (8, 1), (16, 2), (4, 4)])
def test_bbs_spmm_equals_library_matmul_and_alg0(G, K):
    rng = np.random.default_rng(40 + G + K)
    N, O, C = 37, 24, 8 * G
    X = rng.standard_normal((N, C)).astype(np.float32)
    W = rng.standard_normal((O, C)).astype(np.float32)
    vals, idx = oracle.bbs_pack(W, G, K)
    Wd = oracle.bbs_unpack(vals, idx, G)
    Y, Yabs = oracle.bbs_spmm_rows(X, vals, idx, G, want_abs=True)
    np.testing.assert_allclose(Y, X.astype(np.float64) @ Wd.astype(np.float64).T, rtol=1e-12, atol=1e-12)
    np.testing.assert_array_equal(Y, oracle.dense_rows(X, Wd))   # same terms, same (ascending) order
    np.testing.assert_allclose(Yabs, np.abs(X.astype(np.float64)) @ np.abs(Wd.astype(np.float64)).T,
                               rtol=1e-12)
    if K == G:
        np.testing.assert_allclose(Y, X.astype(np.float64) @ W.astype(np.float64).T, rtol=1e-12, atol=1e-12)
    rows = np.array([N - 1, 0, 5], np.int64)
    np.testing.assert_array_equal(oracle.bbs_spmm_rows(X, vals, idx, G, rows=rows), Y[rows])


def test_bbs_index_selects_the_input_inside_its_group():
    """Sec. 3.3: the index of a kept weight picks the input element inside the
    group.  A hand example in exact integers: row 0 keeps inputs 1 and 2 of
    group 0 (|-3| and |2| of [0.25, -3, 2, 0.5]) and inputs 4 and 7 of group 1."""
    W = np.array([[0.25, -3.0, 2.0, 0.5, 5.0, 1.0, -1.0, 4.0]], np.float32)
    vals, idx = oracle.bbs_pack(W, 4, 2)
    assert idx[0].tolist() == [[1, 2], [0, 3]]
    assert vals[0].tolist() == [[-3.0, 2.0], [5.0, 4.0]]
    X = np.array([[1, 10, 100, 1000, 2, 20, 200, 2000]], np.float32)
    Y = oracle.bbs_spmm_rows(X, vals, idx, 4)
    assert Y[0, 0] == -3 * 10 + 2 * 100 + 5 * 2 + 4 * 2000
    # a one-hot input reaches exactly the rows whose kept index names it
    rng = np.random.default_rng(9)
    Wr = rng.standard_normal((6, 8)).astype(np.float32)
    v, i = oracle.bbs_pack(Wr, 4, 2)
    for c in range(8):
        x = np.zeros((1, 8), np.float32)
        x[0, c] = 1.0
        y = oracle.bbs_spmm_rows(x, v, i, 4)[0]
        j, r = divmod(c, 4)
        want = [v[o, j][list(i[o, j]).index(r)] if r in i[o, j] else 0.0 for o in range(6)]
        np.testing.assert_array_equal(y, np.array(want, np.float64))


def test_bbs_spmm_epilogue():
    rng = np.random.default_rng(11)
    N, O, C, G, K = 9, 8, 16, 4, 2
    X = rng.standard_normal((N, C)).astype(np.float32)
    vals, idx = oracle.bbs_pack(rng.standard_normal((O, C)).astype(np.float32), G, K)
    sc = rng.random(O).astype(np.float32) + 0.5
    bi = rng.standard_normal(O).astype(np.float32)
    res = rng.standard_normal((N, O)).astype(np.float32)
    base = oracle.bbs_spmm_rows(X, vals, idx, G)
    y = oracle.bbs_spmm_rows(X, vals, idx, G, scale=sc, bias=bi, residual=res, relu=True)
    np.testing.assert_allclose(y, np.maximum(base * sc + bi + res, 0.0), rtol=1e-12, atol=1e-12)
