"""Pins for the oracle's improved-targeted-dropout functions (Sec. 5.1, the
schedule of Sec. 6) and the gradient of the packed values: hand values of the
ramp, the end of the ramp equal to the CCI projection, a brute-force
candidate set, the dropout rate as a binomial frequency, the threshold edge,
and the gradient against numpy matmul and torch autograd in float64."""
import numpy as np
import pytest
import torch

import oracle
from test_oracle import brute_force_keep


def test_schedule_hand_values():
    # G = 8, K = 2 (75% sparse), 100 steps: first half ramps the candidate
    # count 0 -> 6 at dropout 1/2, second half ramps dropout 1/2 -> 1
    got = [oracle.td_schedule(s, 100, 8, 2) for s in (0, 10, 25, 50, 60, 75, 100)]
    assert got == [(0, 0.5), (1, 0.5), (3, 0.5), (6, 0.5), (6, 0.6), (6, 0.75), (6, 1.0)]
    assert oracle.td_schedule(0, 1, 16, 16) == (0, 0.5)       # K = G: nothing is ever a candidate
    assert oracle.td_schedule(1, 1, 16, 1) == (15, 1.0)


def test_schedule_is_monotone_and_phased():
    T, G, K = 97, 16, 4
    prev = (-1, 0.0)
    for s in range(T + 1):
        n, p = oracle.td_schedule(s, T, G, K)
        assert n >= prev[0] and p >= prev[1]
        if 2 * s < T:
            assert p == 0.5 and n <= G - K
        else:
            assert n == G - K
        prev = (n, p)
    with pytest.raises(ValueError):
        oracle.td_schedule(T + 1, T, G, K)


@pytest.mark.parametrize("G,K", [(4, 2), (8, 2), (16, 1), (8, 8)])
def test_end_of_ramp_is_the_cci_projection(G, K):
    rng = np.random.default_rng(G + K)
    O, C = 4 * G, 33
    W = rng.standard_normal((O, C)).astype(np.float32)
    n, p = oracle.td_schedule(10, 10, G, K)
    bits = rng.integers(0, 2**32, size=(O, C), dtype=np.uint64).astype(np.uint32)
    We, keep = oracle.td_mask(W, G, n, bits, p)
    Wp = oracle.unpack(*oracle.pack(W, G, K), G)
    np.testing.assert_array_equal(We, Wp)
    kept = np.zeros((O, C), np.uint8)
    _, idx = oracle.pack(W, G, K)
    for g in range(O // G):
        for k in range(K):
            kept[g * G + idx[g, k], np.arange(C)] = 1
    np.testing.assert_array_equal(keep, kept)


def test_nothing_dropped_without_candidates_or_rate():
    rng = np.random.default_rng(2)
    W = rng.standard_normal((16, 20)).astype(np.float32)
    bits = np.zeros((16, 20), np.uint32)
    for n, p in ((0, 1.0), (6, 0.0)):
        We, keep = oracle.td_mask(W, 8, n, bits, p)
        np.testing.assert_array_equal(We, W)
        assert keep.all()


@pytest.mark.parametrize("G,n_t", [(4, 1), (8, 3), (8, 7), (6, 2)])
def test_candidates_match_brute_force(G, n_t):
    rng = np.random.default_rng(10 * G + n_t)
    O, C = 3 * G, 15
    W = rng.standard_normal((O, C)).astype(np.float32)
    We, keep = oracle.td_mask(W, G, n_t, np.zeros((O, C), np.uint32), 1.0)   # every candidate dropped
    for g in range(O // G):
        for c in range(C):
            protected = set(brute_force_keep(W[g * G:(g + 1) * G, c], G - n_t))
            for r in range(G):
                assert keep[g * G + r, c] == (1 if r in protected else 0)


def test_dropout_frequency_and_threshold_edge():
    rng = np.random.default_rng(4)
    O, C, G, K = 64, 4096, 8, 2
    W = rng.standard_normal((O, C)).astype(np.float32)
    bits = rng.integers(0, 2**32, size=(O, C), dtype=np.uint64).astype(np.uint32)
    We, keep = oracle.td_mask(W, G, G - K, bits, 0.5)
    cand = 1 - oracle.td_mask(W, G, G - K, np.zeros((O, C), np.uint32), 1.0)[1]
    n = int(cand.sum())
    assert n == O * C * (G - K) // G
    dropped = int((1 - keep)[cand == 1].sum())
    assert abs(dropped / n - 0.5) < 4 * np.sqrt(0.25 / n)       # binomial, 4 sigma
    assert (keep[cand == 0] == 1).all()
    # dropped iff bits < floor(p * 2^32)
    thr = 2**30                                                   # p = 1/4
    b = np.full((8, 1), thr, np.uint32)
    b[3, 0] = thr - 1
    Wt = np.arange(1, 9, dtype=np.float32).reshape(8, 1)          # rows 0..5 are the 6 candidates
    _, kp = oracle.td_mask(Wt, 8, 6, b, 0.25)
    assert kp[:, 0].tolist() == [1, 1, 1, 0, 1, 1, 1, 1]


@pytest.mark.parametrize("G,K", [(8, 2), (16, 1), (4, 4)])
def test_grad_packed_matches_matmul_and_autograd(G, K):
    rng = np.random.default_rng(30 + G + K)
    N, O, C = 19, 2 * G, 24
    X = rng.standard_normal((N, C)).astype(np.float32)
    dY = rng.standard_normal((N, O)).astype(np.float32)
    vals, idx = oracle.pack(rng.standard_normal((O, C)).astype(np.float32), G, K)
    dv = oracle.grad_packed(dY, X, idx, G)
    full = dY.astype(np.float64).T @ X.astype(np.float64)            # dL/dW_hat [O, C]
    rows = (np.arange(O // G)[:, None, None] * G + idx).astype(np.int64)
    np.testing.assert_allclose(dv, full[rows, np.arange(C)[None, None, :]], rtol=1e-12, atol=1e-12)
    # autograd of L = sum(dY * (X W_hat^T)) with W_hat scattered from the packed values
    v = torch.from_numpy(vals.astype(np.float64)).requires_grad_(True)
    Wh = torch.zeros((O, C), dtype=torch.float64)
    Wh = Wh.index_put((torch.from_numpy(rows.reshape(-1)), torch.arange(C).repeat(O // G * K)), v.reshape(-1))
    L = (torch.from_numpy(dY).double() * (torch.from_numpy(X).double() @ Wh.T)).sum()
    L.backward()
    np.testing.assert_allclose(dv, v.grad.numpy(), rtol=1e-12, atol=1e-12)
