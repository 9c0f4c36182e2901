"""Full-size parity: every output of the benchmark configurations against the
oracle (Alg. 1 / the direct convolution in double precision).

  - 3x3 conv, batch 32, 56x56, 64 -> 64, G=8, K=2: all 100,352 x 64 outputs;
  - 1x1 bottleneck conv, batch 64, 14x14, 1024 -> 256, G=16, K=4 and K=2: all
    12,544 x 256 outputs;
  - 4096^3 FC, G=16, K in {1, 2, 4, 8, 16}: all 4096 x 4096 outputs;

each through every kernel family that takes the shape, writing into a
sentinel-guarded buffer.  The oracle result of a configuration is computed
once and shared by the families.
"""
import functools

import numpy as np
import pytest
import torch

import oracle
from gpu_common import DEV, Guarded, need_gpu, oracle_pack_vals, x_as_f32
from parity import TOL, check_close, to_np_f32
from paper_1910_11971_amd import workloads

pytestmark = pytest.mark.gpu


@functools.lru_cache(maxsize=1)
def reference(name):
    """(X, W, oracle Y, oracle sum of |terms|) of a workload, every output."""
    wl = workloads.WORKLOADS[name]
    X, W = workloads.draw(wl)
    v_ref, idx_ref, _ = oracle_pack_vals(W, wl.G, wl.K, torch.bfloat16)
    if wl.conv:
        Wm = oracle.unpack(v_ref, idx_ref, wl.G).reshape(wl.O, wl.KH, wl.KW, wl.Cin)
        Y, Yabs = oracle.conv2d_nhwc(x_as_f32(X), Wm, (wl.stride,) * 2, (wl.pad,) * 2, want_abs=True)
    else:
        Y, Yabs = oracle.spmm_rows(x_as_f32(X), v_ref, idx_ref, wl.G, want_abs=True)
    return X, W, Y, Yabs


def run_full(name, algo):
    from paper_1910_11971_amd import cci
    wl = workloads.WORKLOADS[name]
    X, W, Yref, Yabs = reference(name)
    print(f"[full-size] {name} {algo}: N={wl.N} C={wl.C} O={wl.O} G={wl.G} K={wl.K}", flush=True)
    vals, idx = cci.pack(torch.from_numpy(W).to(DEV), wl.G, wl.K, torch.bfloat16)
    Xd = X.to(DEV)
    if wl.conv:
        Yg = Guarded((wl.B, wl.Ho, wl.Wo, wl.O), torch.bfloat16)
        cci.conv_im2col(Xd, vals, idx, wl.G, wl.KH, wl.KW, (wl.stride,) * 2, (wl.pad,) * 2,
                        out_dtype=torch.bfloat16, algo=algo, out=Yg.t)
    else:
        Yg = Guarded((wl.N, wl.O), torch.bfloat16)
        cci.spmm(Xd, vals, idx, wl.G, out_dtype=torch.bfloat16, algo=algo, out=Yg.t)
    torch.cuda.synchronize()
    Yg.check(f"{name} {algo}")
    got = to_np_f32(Yg.t).reshape(wl.N, wl.O)
    assert got.size == Yref.size == wl.N * wl.O
    check_close(got, Yref, Yabs, TOL["bf16"], f"{name} {algo} (all {wl.N * wl.O} outputs)")


@pytest.mark.parametrize("algo", ["auto", "resident_mfma", "dense_tile_mfma", "sparse_mac"])
def test_conv3x3_every_output(algo):
    need_gpu()
    run_full("conv3x3", algo)


@pytest.mark.parametrize("name,algo", [(n, a) for n in ("conv1x1_k4", "conv1x1_k2")
                                       for a in ("auto", "tap_tile_mfma", "wide_tile_mfma", "dense_tile_mfma",
                                                 "sparse_mac")])
def test_conv1x1_bottleneck_every_output(name, algo):
    need_gpu()
    run_full(name, algo)


@pytest.mark.parametrize("K,algo", [(k, a) for k in (1, 2, 4, 8, 16)
                                    for a in ("auto", "wide_tile_mfma", "tap_tile_mfma", "dense_tile_mfma",
                                              "sparse_mac")])
def test_fc4096_every_output(K, algo):
    need_gpu()
    run_full(f"fc4096_k{K}", algo)
