"""cci_pack on the GPU vs the oracle: indices and values bit-exact."""
import numpy as np
import pytest
import torch

from gpu_common import DEV, Guarded, gpu_bits, need_gpu, oracle_pack_vals
from paper_1910_11971_amd import workloads

pytestmark = pytest.mark.gpu


def run_pack(W: np.ndarray, G, K, vdt):
    from paper_1910_11971_amd import cci
    Wt = torch.from_numpy(W).to(DEV)
    O, C = W.shape
    vg, ig = Guarded((O // G, K, C), vdt), Guarded((O // G, K, C), torch.uint8)
    vals, idx = cci.pack(Wt, G, K, vdt, out=(vg.t, ig.t))
    torch.cuda.synchronize()
    vg.check(f"pack vals O={O} C={C} G={G} K={K}")
    ig.check(f"pack idx O={O} C={C} G={G} K={K}")
    _, idx_ref, bits_ref = oracle_pack_vals(W, G, K, vdt)
    np.testing.assert_array_equal(idx.cpu().numpy(), idx_ref)
    np.testing.assert_array_equal(gpu_bits(vals), bits_ref)


@pytest.mark.parametrize("vdt", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("O,C,G,K", [
    (256, 256, 8, 4), (64, 576, 8, 2), (256, 1024, 16, 4), (256, 1024, 16, 2),
    (32, 300, 2, 1), (32, 257, 4, 3), (64, 513, 32, 5), (64, 77, 16, 16), (64, 1, 8, 1),
    (48, 37, 6, 2), (96, 130, 3, 2), (128, 40, 64, 9), (512, 33, 256, 7), (256, 5, 256, 256),
])
def test_pack_matches_oracle(O, C, G, K, vdt):
    need_gpu()
    rng = np.random.default_rng(O * 1000 + C + G + K)
    W = rng.standard_normal((O, C)).astype(np.float32)
    run_pack(W, G, K, vdt)


@pytest.mark.parametrize("vdt", [torch.float32, torch.bfloat16])
def test_pack_ties_zeros_and_specials(vdt):
    need_gpu()
    rng = np.random.default_rng(5)
    W = rng.choice(np.array([0.0, -0.0, 1.0, -1.0, 0.5, -0.5, 2.0], np.float32), size=(64, 200))
    W[0, :5] = [np.inf, -np.inf, np.nan, 3e38, -1e-40]
    run_pack(W.astype(np.float32), 8, 3, vdt)
    run_pack(W.astype(np.float32), 16, 5, vdt)
    # selection from the top (K <= G / 2) and from the bottom, on heavy ties
    for G, K in ((16, 1), (16, 2), (16, 4), (16, 7), (16, 8), (16, 12), (8, 1), (8, 6), (4, 1), (32, 3), (32, 24)):
        run_pack(W.astype(np.float32), G, K, vdt)


@pytest.mark.parametrize("vdt", [torch.float32, torch.bfloat16])
def test_pack_near_ties(vdt):
    # |w| that agree above their last few mantissa bits (columns the kernel re-ranks exactly),
    # exact ties, and both ends of the selection (K <= G / 2 from the top, K > G / 2 from the bottom)
    need_gpu()
    rng = np.random.default_rng(11)
    base = rng.standard_normal((1, 300)).astype(np.float32).view(np.uint32)
    low = rng.integers(0, 64, size=(64, 300)).astype(np.uint32)
    W = ((base & np.uint32(0xffffffc0)) | low).view(np.float32)
    W = W * rng.choice(np.array([1.0, -1.0], np.float32), size=W.shape)
    W[:, ::7] = W[0:1, ::7]
    for G, K in ((2, 1), (4, 1), (4, 3), (8, 3), (8, 5), (16, 1), (16, 4), (16, 8), (16, 9), (16, 15),
                 (32, 1), (32, 7), (32, 16), (32, 20), (32, 31)):
        run_pack(np.ascontiguousarray(W), G, K, vdt)


@pytest.mark.parametrize("K", [1, 2, 4, 8, 16])
def test_pack_full_size_fc4096(K):
    need_gpu()
    _, W = workloads.draw(workloads.WORKLOADS[f"fc4096_k{K}"])
    run_pack(W, 16, K, torch.bfloat16)


@pytest.mark.parametrize("name", ["fc256", "conv3x3", "conv1x1_k4", "conv1x1_k2"])
def test_pack_full_size_configs(name):
    need_gpu()
    wl = workloads.WORKLOADS[name]
    _, W = workloads.draw(wl)
    run_pack(W, wl.G, wl.K, torch.float32 if wl.x_dtype == "f32" else torch.bfloat16)
