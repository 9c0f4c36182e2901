"""Balanced sparsity and the 2:4 sparse matrix-core product on the GPU against
the oracle: the balanced projection bit for bit, the prepared 2:4 operand
decoded from its documented layout, the balanced-sparse product, and the
backward product dX = dY . W_hat of a CCI layer through the 2:4 operand of
W_hat^T."""
import functools

import numpy as np
import pytest
import torch

import oracle
from gpu_common import DEV, Guarded, gpu_bits, need_gpu
from parity import TOL, check_close, to_np_f32

pytestmark = pytest.mark.gpu


def bf16_vals(v32):
    return oracle.bf16_bits_to_f32(oracle.bf16_rne(v32))


def decode_2of4(av: torch.Tensor, ai: torch.Tensor) -> np.ndarray:
    """Dense [M, R] matrix of a prepared 2:4 operand, read from the layout the
    header documents: lane l of fragment (s, mb) is row 16 mb + l % 16 and
    columns 64 s + 16 (l / 16) + 4 (e / 2) + bits 2e..2e+1 of its index."""
    v = av.float().cpu().numpy()                                        # [S, MB, 64, 8]
    w = ai.cpu().numpy().view(np.uint16).astype(np.int64)               # [S, MB, 64]
    S, MB = v.shape[:2]
    A = np.zeros((MB * 16, S * 64), np.float64)
    s, mb, l, e = np.meshgrid(np.arange(S), np.arange(MB), np.arange(64), np.arange(8), indexing="ij")
    z = (w[s, mb, l] >> (2 * e)) & 3
    rows = mb * 16 + l % 16
    cols = 64 * s + 16 * (l // 16) + 4 * (e // 2) + z
    np.add.at(A, (rows.ravel(), cols.ravel()), v.ravel())
    # each 4-run holds two distinct positions (unused slots get one of their own)
    z2 = z.reshape(S, MB, 64, 4, 2)
    assert (z2[..., 0] != z2[..., 1]).all()
    return A


def rand(shape, seed, scale=1.0):
    return (np.random.default_rng(seed).standard_normal(shape) * scale).astype(np.float32)


# ------------------------------------------------------------------ pack ----

@pytest.mark.parametrize("vdt", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("O,C,G,K", [(64, 256, 4, 2), (33, 96, 8, 3), (16, 4096, 16, 1), (8, 512, 256, 7),
                                     (5, 40, 2, 1), (128, 192, 16, 16), (7, 60, 5, 2)])
def test_bbs_pack_matches_oracle(O, C, G, K, vdt):
    need_gpu()
    from paper_1910_11971_amd import cci
    W = rand((O, C), O + C + G)
    W[0, :4] = [np.inf, -0.0, np.nan, -3e38]
    W[1, :G] = 1.0   # ties inside a group: lower position wins
    vg, ig = Guarded((O, C // G, K), vdt), Guarded((O, C // G, K), torch.uint8)
    cci.bbs_pack(torch.from_numpy(W).to(DEV), G, K, vdt, out=(vg.t, ig.t))
    torch.cuda.synchronize()
    vg.check("bbs vals")
    ig.check("bbs idx")
    v32, ix = oracle.bbs_pack(W, G, K)
    np.testing.assert_array_equal(ig.t.cpu().numpy(), ix)
    ref_bits = oracle.bf16_rne(v32) if vdt == torch.bfloat16 else v32.view(np.uint32)
    np.testing.assert_array_equal(gpu_bits(vg.t), ref_bits)


# -------------------------------------------------------- 2:4 operands ------

@pytest.mark.parametrize("O,C,G,K", [(16, 64, 4, 2), (48, 192, 4, 1), (32, 128, 8, 2), (32, 128, 8, 1),
                                     (64, 256, 16, 2), (16, 256, 16, 1), (16, 256, 32, 2), (16, 128, 64, 1)])
def test_bbs_to_2of4_decodes_to_the_masked_matrix(O, C, G, K):
    need_gpu()
    from paper_1910_11971_amd import cci
    W = rand((O, C), 3 * O + G + K)
    vals, idx = cci.bbs_pack(torch.from_numpy(W).to(DEV), G, K)
    av, ai = cci.bbs_to_2of4(vals, idx, G)
    torch.cuda.synchronize()
    v32, ix = oracle.bbs_pack(W, G, K)
    np.testing.assert_array_equal(decode_2of4(av, ai), oracle.bbs_unpack(bf16_vals(v32), ix, G))


@pytest.mark.parametrize("O,C,G,K", [(64, 16, 4, 2), (128, 48, 8, 1), (64, 32, 16, 2), (256, 16, 32, 2)])
def test_cci_to_2of4_transposed_decodes_to_the_transpose(O, C, G, K):
    need_gpu()
    from paper_1910_11971_amd import cci
    W = rand((O, C), O + 5 * C + K)
    vals, idx = cci.pack(torch.from_numpy(W).to(DEV), G, K, torch.bfloat16)
    av, ai = cci.to_2of4_transposed(vals, idx, G)
    torch.cuda.synchronize()
    v32, ix = oracle.pack(W, G, K)
    np.testing.assert_array_equal(decode_2of4(av, ai), oracle.unpack(bf16_vals(v32), ix, G).T)


# ------------------------------------------------------ 2:4 products -------

def run_bbs(N, O, C, G, K, y_dtype=torch.bfloat16, ep=False, seed=0, X=None, W=None):
    from paper_1910_11971_amd import cci
    X = rand((N, C), seed + 1) if X is None else X
    W = rand((O, C), seed + 2, 1 / np.sqrt(C)) if W is None else W
    Xt = torch.from_numpy(X).to(torch.bfloat16)
    vals, idx = cci.bbs_pack(torch.from_numpy(W).to(DEV), G, K)
    av, ai = cci.bbs_to_2of4(vals, idx, G)
    kw, s, b, r = {}, None, None, None
    if ep:
        rng = np.random.default_rng(seed + 3)
        s = (0.5 + rng.random(O)).astype(np.float32)
        b = (0.1 * rng.standard_normal(O)).astype(np.float32)
        r_t = torch.from_numpy(rng.standard_normal((N, O)).astype(np.float32)).to(y_dtype)
        r = r_t.float().numpy()
        kw = dict(scale=torch.from_numpy(s).to(DEV), bias=torch.from_numpy(b).to(DEV), residual=r_t.to(DEV),
                  relu=True)
    Yg = Guarded((N, O), y_dtype)
    cci.spmm_2of4(Xt.to(DEV), av, ai, out_dtype=y_dtype, out=Yg.t, **kw)
    torch.cuda.synchronize()
    Yg.check(f"bbs N={N} O={O} C={C} G={G} K={K}")
    v32, ix = oracle.bbs_pack(W, G, K)
    Yref, Yabs = oracle.bbs_spmm_rows(Xt.float().numpy(), bf16_vals(v32), ix, G, scale=s, bias=b, residual=r,
                                      relu=ep, want_abs=True)
    S = Yabs.copy()
    if ep:
        S = S * np.abs(s)[None, :] + np.abs(b)[None, :] + np.abs(r)
    tol = TOL["bf16"]
    check_close(to_np_f32(Yg.t), Yref, S, tol, f"bbs 2:4 N={N} O={O} C={C} G={G} K={K}")


@pytest.mark.parametrize("N,O,C,G,K", [
    (1, 16, 64, 4, 2), (37, 48, 128, 4, 2), (300, 272, 192, 4, 1), (1000, 256, 576, 8, 2),
    (257, 512, 256, 16, 1), (513, 784, 320, 16, 2), (64, 32, 1024, 32, 2), (2048, 256, 64, 4, 2),
])
def test_bbs_product(N, O, C, G, K):
    need_gpu()
    run_bbs(N, O, C, G, K, seed=N + O)


@pytest.mark.parametrize("y_dtype", [torch.bfloat16, torch.float32])
def test_bbs_product_epilogue(y_dtype):
    need_gpu()
    run_bbs(333, 96, 256, 4, 2, y_dtype=y_dtype, ep=True, seed=7)


@pytest.mark.parametrize("G,K", [(4, 2), (16, 1), (16, 2)])
def test_bbs_product_fc4096_every_output(G, K):
    """The 4096^3 FC shape of the sparsity sweep with balanced groups."""
    need_gpu()
    from paper_1910_11971_amd import workloads
    X, W = workloads.draw(workloads.WORKLOADS["fc4096_k1"])
    run_bbs(4096, 4096, 4096, G, K, X=X.float().numpy(), W=W)


def run_cci_backward(N, O, C, G, K, seed=0, dY=None, W=None, y_dtype=torch.bfloat16):
    """dX [N, C] = dY [N, O] . W_hat through the 2:4 operand of W_hat^T."""
    from paper_1910_11971_amd import cci
    dY = rand((N, O), seed + 1) if dY is None else dY
    W = rand((O, C), seed + 2, 1 / np.sqrt(O)) if W is None else W
    dYt = torch.from_numpy(dY).to(torch.bfloat16)
    vals, idx = cci.pack(torch.from_numpy(W).to(DEV), G, K, torch.bfloat16)
    av, ai = cci.to_2of4_transposed(vals, idx, G)
    Xg = Guarded((N, C), y_dtype)
    cci.spmm_2of4(dYt.to(DEV), av, ai, out_dtype=y_dtype, out=Xg.t)
    torch.cuda.synchronize()
    Xg.check(f"dX N={N} O={O} C={C}")
    v32, ix = oracle.pack(W, G, K)
    Wm = oracle.unpack(bf16_vals(v32), ix, G)                          # W_hat [O, C]
    d = dYt.float().numpy()
    ref = oracle.dense_rows(d, np.ascontiguousarray(Wm.T))              # sum_o dY[n][o] W_hat[o][c]
    terms = np.abs(d.astype(np.float64)) @ np.abs(Wm.astype(np.float64))
    check_close(to_np_f32(Xg.t), ref, terms, TOL["bf16"], f"cci backward dX N={N} O={O} C={C} G={G} K={K}")


@pytest.mark.parametrize("N,O,C,G,K", [(1, 64, 16, 4, 2), (300, 128, 48, 8, 1), (999, 256, 272, 16, 2),
                                       (64, 576, 64, 8, 2), (2000, 192, 512, 4, 1)])
def test_cci_backward_data(N, O, C, G, K):
    need_gpu()
    run_cci_backward(N, O, C, G, K, seed=N + C, y_dtype=torch.float32 if N == 999 else torch.bfloat16)


@pytest.mark.parametrize("K", [1, 2])
def test_cci_backward_data_fc4096_every_output(K):
    need_gpu()
    from paper_1910_11971_amd import workloads
    X, W = workloads.draw(workloads.WORKLOADS[f"fc4096_k{K}"])
    run_cci_backward(4096, 4096, 4096, 16, K, dY=X.float().numpy(), W=W)


def test_2of4_rejects_what_it_cannot_hold():
    need_gpu()
    from paper_1910_11971_amd import cci
    W = torch.from_numpy(rand((32, 128), 1)).to(DEV)
    vals, idx = cci.bbs_pack(W, 8, 3)   # a run of 4 inputs may hold 3 kept weights
    with pytest.raises(cci.CCIError):
        cci.bbs_to_2of4(vals, idx, 8)
    v2, i2 = cci.bbs_pack(W, 4, 2, torch.float32)   # fp32 values
    with pytest.raises(cci.CCIError):
        cci.bbs_to_2of4(v2, i2, 4)
