"""Improved targeted dropout on the GPU against the oracle: candidate dropout
of one step (bit for bit), the gradient of the packed values, and one whole
training step at the end of the ramp (mask, re-projection, forward, backward
data and packed-value gradient)."""
import numpy as np
import pytest
import torch

import oracle
from gpu_common import DEV, Guarded, gpu_bits, need_gpu
from parity import TOL, check_close, to_np_f32

pytestmark = pytest.mark.gpu


def rand_bits(shape, seed):
    return np.random.default_rng(seed).integers(0, 2**32, size=shape, dtype=np.uint64).astype(np.uint32)


def run_mask(W, G, n_t, bits, p, wdt):
    from paper_1910_11971_amd import cci
    O, C = W.shape
    wg, kg = Guarded((O, C), wdt), Guarded((O, C), torch.uint8)
    cci.td_mask(torch.from_numpy(W).to(DEV), G, n_t, torch.from_numpy(bits.view(np.int32)).to(DEV), p, wdt,
                out=(wg.t, kg.t))
    torch.cuda.synchronize()
    wg.check("W_eff")
    kg.check("keep")
    We, keep = oracle.td_mask(W, G, n_t, bits, p)
    np.testing.assert_array_equal(kg.t.cpu().numpy(), keep)
    ref_bits = oracle.bf16_rne(We) if wdt == torch.bfloat16 else We.view(np.uint32)
    np.testing.assert_array_equal(gpu_bits(wg.t), ref_bits)


@pytest.mark.parametrize("wdt", [torch.bfloat16, torch.float32])
@pytest.mark.parametrize("O,C,G,n_t,p", [(64, 300, 8, 3, 0.5), (64, 300, 8, 6, 1.0), (48, 129, 16, 15, 0.75),
                                         (32, 1000, 4, 2, 0.0), (64, 77, 32, 20, 0.6), (36, 50, 6, 4, 0.5),
                                         (256, 40, 256, 200, 0.9), (16, 4096, 16, 0, 1.0)])
def test_td_mask_matches_oracle(O, C, G, n_t, p, wdt):
    need_gpu()
    rng = np.random.default_rng(O + C + G + n_t)
    W = rng.standard_normal((O, C)).astype(np.float32)
    W[:G, 0] = 1.0                                   # a tied group
    W[0, 1:4] = [np.inf, -0.0, -3e38]
    run_mask(W, G, n_t, rand_bits((O, C), n_t + 1), p, wdt)


def test_td_mask_threshold_edge_and_end_of_ramp():
    need_gpu()
    W = np.arange(1, 9, dtype=np.float32).reshape(8, 1).repeat(64, axis=1)
    bits = np.full((8, 64), 2**30, np.uint32)
    bits[3, :] = 2**30 - 1
    run_mask(W, 8, 6, bits, 0.25, torch.float32)     # only row 3 (a candidate below the threshold) drops
    from paper_1910_11971_amd import cci
    rng = np.random.default_rng(3)
    W = rng.standard_normal((128, 512)).astype(np.float32)
    n, p = cci.td_schedule(100, 100, 8, 2)
    We, keep = cci.td_mask(torch.from_numpy(W).to(DEV), 8, n, torch.from_numpy(rand_bits(W.shape, 5).view(np.int32)).to(DEV),
                           p, torch.float32)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(We.cpu().numpy(), oracle.unpack(*oracle.pack(W, 8, 2), 8))


def run_grad(N, O, C, G, K, dt, seed=0, dY=None, X=None, W=None):
    from paper_1910_11971_amd import cci
    rng = np.random.default_rng(seed)
    dY = rng.standard_normal((N, O)).astype(np.float32) if dY is None else dY
    X = rng.standard_normal((N, C)).astype(np.float32) if X is None else X
    W = rng.standard_normal((O, C)).astype(np.float32) if W is None else W
    dYt = torch.from_numpy(dY).to(dt)
    Xt = torch.from_numpy(X).to(dt)
    _, idx = cci.pack(torch.from_numpy(W).to(DEV), G, K, torch.float32)
    dg = Guarded((O // G, K, C), torch.float32)
    cci.grad_packed(dYt.to(DEV), Xt.to(DEV), idx, G, out=dg.t)
    torch.cuda.synchronize()
    dg.check("dvals")
    _, ix = oracle.pack(W, G, K)
    np.testing.assert_array_equal(idx.cpu().numpy(), ix)
    d, x = dYt.float().numpy(), Xt.float().numpy()
    ref = oracle.grad_packed(d, x, ix, G)
    rows = (np.arange(O // G)[:, None, None] * G + ix).astype(np.int64)
    terms = (np.abs(d.astype(np.float64)).T @ np.abs(x.astype(np.float64)))[rows, np.arange(C)[None, None, :]]
    tol = TOL["f32"] if dt == torch.float32 else TOL["bf16"]
    check_close(to_np_f32(dg.t), ref, terms, tol, f"grad_packed N={N} O={O} C={C} G={G} K={K}")


@pytest.mark.parametrize("N,O,C,G,K", [(1, 16, 64, 8, 2), (100, 64, 300, 8, 3), (257, 128, 1000, 16, 1),
                                       (64, 64, 256, 4, 4), (130, 64, 70, 32, 9), (65, 512, 40, 256, 17),
                                       (300, 96, 129, 16, 16), (0, 16, 64, 8, 2)])
@pytest.mark.parametrize("dt", [torch.bfloat16, torch.float32])
def test_grad_packed_matches_oracle(N, O, C, G, K, dt):
    need_gpu()
    run_grad(N, O, C, G, K, dt, seed=N + C + K)


@pytest.mark.parametrize("N,O,C,G,K", [(96, 264, 520, 8, 3), (33, 1024, 64, 128, 5), (200, 256, 256, 1, 1),
                                       (64, 136, 8, 2, 2), (500, 64, 2056, 64, 64), (32, 512, 768, 16, 4),
                                       (1000, 40, 24, 4, 1)])
def test_grad_packed_matrix_cores(N, O, C, G, K):
    """bf16 shapes the matrix-core kernel takes: ragged sample steps, partial 256 x 256 tiles, G from 1 to 128,
    K = G (dense control)."""
    need_gpu()
    run_grad(N, O, C, G, K, torch.bfloat16, seed=N + O + C + K)


@pytest.mark.parametrize("K", [1, 4])
def test_grad_packed_fc4096_every_output(K):
    need_gpu()
    from paper_1910_11971_amd import workloads
    X, W = workloads.draw(workloads.WORKLOADS[f"fc4096_k{K}"])
    dY = np.random.default_rng(9).standard_normal((4096, 4096)).astype(np.float32)
    run_grad(4096, 4096, 4096, 16, K, torch.bfloat16, dY=dY, X=X.float().numpy(), W=W)


def test_training_step_at_the_end_of_the_ramp():
    """mask (every candidate dropped) == re-projection; forward, dX and the
    packed-value gradient of the fixed-mask layer, each against the oracle."""
    need_gpu()
    from paper_1910_11971_amd import cci
    rng = np.random.default_rng(21)
    N, O, C, G, K = 512, 256, 320, 8, 2
    W = (rng.standard_normal((O, C)) / np.sqrt(C)).astype(np.float32)
    X = torch.from_numpy(rng.standard_normal((N, C)).astype(np.float32)).to(torch.bfloat16)
    dY = torch.from_numpy(rng.standard_normal((N, O)).astype(np.float32)).to(torch.bfloat16)
    Wd = torch.from_numpy(W).to(DEV)
    n, p = cci.td_schedule(1000, 1000, G, K)
    We, keep = cci.td_mask(Wd, G, n, torch.from_numpy(rand_bits((O, C), 2).view(np.int32)).to(DEV), p, torch.float32)
    vals, idx = cci.pack(Wd, G, K, torch.bfloat16)
    Y = cci.spmm(X.to(DEV), vals, idx, G)
    tv, ti = cci.to_2of4_transposed(vals, idx, G)
    dX = cci.spmm_2of4(dY.to(DEV), tv, ti)
    dv = cci.grad_packed(dY.to(DEV), X.to(DEV), idx, G)
    torch.cuda.synchronize()
    v32, ix = oracle.pack(W, G, K)
    np.testing.assert_array_equal(We.cpu().numpy(), oracle.unpack(v32, ix, G))
    np.testing.assert_array_equal(keep.cpu().numpy(), (oracle.unpack(v32, ix, G) != 0).astype(np.uint8))
    vb = oracle.bf16_bits_to_f32(oracle.bf16_rne(v32))
    Wm = oracle.unpack(vb, ix, G)
    x, d = X.float().numpy(), dY.float().numpy()
    y_ref, y_abs = oracle.spmm_rows(x, vb, ix, G, want_abs=True)
    check_close(to_np_f32(Y), y_ref, y_abs, TOL["bf16"], "forward")
    check_close(to_np_f32(dX), oracle.dense_rows(d, np.ascontiguousarray(Wm.T)), np.abs(d) @ np.abs(Wm),
                TOL["bf16"], "dX")
    rows = (np.arange(O // G)[:, None, None] * G + ix).astype(np.int64)
    terms = (np.abs(d.astype(np.float64)).T @ np.abs(x.astype(np.float64)))[rows, np.arange(C)[None, None, :]]
    check_close(to_np_f32(dv), oracle.grad_packed(d, x, ix, G), terms, TOL["bf16"], "dvals")
