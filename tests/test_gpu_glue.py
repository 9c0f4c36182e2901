"""CNN glue kernels vs the oracle: max pooling exact, average pooling to tol."""
import numpy as np
import pytest
import torch

import oracle
from gpu_common import DEV, need_gpu
from parity import to_np_f32

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("dt", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("shape,k,s,p", [((2, 112, 112, 64), 3, 2, 1), ((3, 9, 10, 5), 3, 2, 1),
                                         ((1, 8, 8, 16), 2, 2, 0), ((2, 13, 11, 24), 3, 2, 1),
                                         ((1, 7, 9, 40), 3, 1, 1)])
def test_maxpool_exact(shape, k, s, p, dt):
    need_gpu()
    from paper_1910_11971_amd import cci
    X = torch.from_numpy(np.random.default_rng(1).standard_normal(shape).astype(np.float32)).to(dt)
    Y = cci.maxpool2d_nhwc(X.to(DEV), k, s, p)
    ref = oracle.maxpool2d_nhwc(X.float().numpy(), k, s, p)
    np.testing.assert_array_equal(to_np_f32(Y), ref)


@pytest.mark.parametrize("shape", [(4, 7, 7, 2048), (3, 5, 6, 12), (2, 9, 11, 40)])
@pytest.mark.parametrize("xdt,ydt", [(torch.bfloat16, torch.bfloat16), (torch.bfloat16, torch.float32),
                                     (torch.float32, torch.float32)])
def test_global_avgpool(xdt, ydt, shape):
    need_gpu()
    from paper_1910_11971_amd import cci
    X = torch.from_numpy(np.random.default_rng(2).standard_normal(shape).astype(np.float32)).to(xdt)
    Y = cci.global_avgpool_nhwc(X.to(DEV), ydt)
    ref = oracle.global_avgpool_nhwc(X.float().numpy())
    tol = 1e-5 if ydt == torch.float32 else 1e-2
    err = np.abs(to_np_f32(Y) - ref).max() / np.abs(ref).max()
    assert err <= tol
