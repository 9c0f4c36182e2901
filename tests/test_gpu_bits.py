"""Plain log2(G)-bit indices on the GPU: the stream bit for bit against the
oracle, and the few-row product reading it (or the byte array) against the
oracle's Alg. 1, with identical results for both index widths."""
import numpy as np
import pytest
import torch

import oracle
from gpu_common import DEV, Guarded, need_gpu
from parity import TOL, check_close, to_np_f32

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("n,G", [(1, 2), (37, 4), (1000, 8), (4096, 16), (777, 64), (96, 256), (33, 3), (130, 6),
                                 (5000, 32), (31, 128)])
def test_index_stream_matches_oracle(n, G):
    need_gpu()
    from paper_1910_11971_amd import cci
    b = cci.index_width(G)
    assert b == oracle.index_width(G)
    idx = np.random.default_rng(n + G).integers(0, G, size=n).astype(np.uint8)
    nbytes = (n * b + 31) // 32 * 4
    wg = Guarded((nbytes // 4,), torch.int32)
    cci.index_bits(torch.from_numpy(idx).to(DEV), b, out=wg.t)
    torch.cuda.synchronize()
    wg.check("index stream")
    np.testing.assert_array_equal(wg.t.cpu().numpy().view(np.uint32), oracle.index_bits(idx, b))


def run_bits(N, C, O, G, K, y_dtype=torch.bfloat16, ep=False, seed=0, X=None, W=None):
    from paper_1910_11971_amd import cci
    rng = np.random.default_rng(seed)
    X = rng.standard_normal((N, C)).astype(np.float32) if X is None else X
    W = (rng.standard_normal((O, C)) / np.sqrt(C)).astype(np.float32) if W is None else W
    Xt = torch.from_numpy(X).to(torch.bfloat16)
    vals, idx = cci.pack(torch.from_numpy(W).to(DEV), G, K, torch.bfloat16)
    b = cci.index_width(G)
    stream = cci.index_bits(idx, b)
    kw, s, bi, r = {}, None, None, None
    if ep:
        s = (0.5 + rng.random(O)).astype(np.float32)
        bi = (0.1 * rng.standard_normal(O)).astype(np.float32)
        r_t = torch.from_numpy(rng.standard_normal((N, O)).astype(np.float32)).to(y_dtype)
        r = r_t.float().numpy()
        kw = dict(scale=torch.from_numpy(s).to(DEV), bias=torch.from_numpy(bi).to(DEV), residual=r_t.to(DEV),
                  relu=True)
    outs = []
    for idx_arg, bits in ((stream, b), (idx, 8)):
        Yg = Guarded((N, O), y_dtype)
        cci.spmm_bits(Xt.to(DEV), vals, idx_arg, G, bits, out_dtype=y_dtype, out=Yg.t, **kw)
        torch.cuda.synchronize()
        Yg.check(f"spmm_bits N={N} C={C} O={O} G={G} K={K} bits={bits}")
        outs.append(Yg.t.clone())
    # the same products in the same order: identical bits whichever index width
    assert torch.equal(outs[0].view(torch.uint8), outs[1].view(torch.uint8))
    v32, ix = oracle.pack(W, G, K)
    vb = oracle.bf16_bits_to_f32(oracle.bf16_rne(v32))
    Yref, Yabs = oracle.spmm_rows(Xt.float().numpy(), vb, ix, G, scale=s, bias=bi, residual=r, relu=ep,
                                  want_abs=True)
    S = Yabs
    if ep:
        S = Yabs * np.abs(s)[None, :] + np.abs(bi)[None, :] + np.abs(r)
    check_close(to_np_f32(outs[0]), Yref, S, TOL["bf16"], f"spmm_bits N={N} C={C} O={O} G={G} K={K}")


@pytest.mark.parametrize("N,C,O,G,K", [
    (1, 32, 16, 8, 2), (5, 96, 48, 4, 1), (16, 256, 64, 16, 4), (17, 320, 96, 2, 1), (40, 64, 32, 32, 5),
    (64, 512, 256, 64, 3), (3, 128, 768, 256, 17), (9, 288, 48, 6, 2), (33, 160, 48, 24, 7), (64, 96, 128, 8, 8),
])
def test_spmm_bits_matches_oracle(N, C, O, G, K):
    need_gpu()
    run_bits(N, C, O, G, K, seed=N + C + G)


@pytest.mark.parametrize("y_dtype", [torch.bfloat16, torch.float32])
def test_spmm_bits_epilogue(y_dtype):
    need_gpu()
    run_bits(20, 256, 128, 8, 2, y_dtype=y_dtype, ep=True, seed=3)


@pytest.mark.parametrize("N,K", [(1, 4), (16, 4), (64, 1)])
def test_spmm_bits_fc4096_every_output(N, K):
    """The 4096 x 4096 layer of the sparsity sweep (G = 16) at decode-sized batches."""
    need_gpu()
    from paper_1910_11971_amd import workloads
    X, W = workloads.draw(workloads.WORKLOADS[f"fc4096_k{K}"])
    run_bits(N, 4096, 4096, 16, K, X=X[:N].float().numpy(), W=W)
