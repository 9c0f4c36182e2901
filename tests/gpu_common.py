"""Shared helpers for GPU parity tests: seeded inputs from the workload
generators, reference values from the CPU oracle, nothing from the HIP path."""
import numpy as np
import pytest
import torch

import oracle
from parity import TOL, bits_u16, check_close, to_np_f32

DEV = "cuda:0"


GUARD_BYTES = 4096   # sentinel bytes on each side of an output buffer
SENTINEL = 0x7F      # bf16 0x7F7F / fp32 0x7F7F7F7F: huge finite values, so an output left unwritten fails too


class Guarded:
    """An output tensor inside a larger device buffer whose margins hold a
    sentinel byte: `check()` asserts that no kernel wrote outside the output
    (the body starts as the sentinel too, so an unwritten element fails the
    value comparison)."""

    def __init__(self, shape, dtype, device=DEV):
        self.nbytes = int(np.prod(shape)) * torch.empty((), dtype=dtype).element_size()
        self.buf = torch.full((self.nbytes + 2 * GUARD_BYTES,), SENTINEL, dtype=torch.uint8, device=device)
        self.t = self.buf[GUARD_BYTES:GUARD_BYTES + self.nbytes].view(dtype).view(shape)

    def check(self, what=""):
        head = self.buf[:GUARD_BYTES]
        tail = self.buf[GUARD_BYTES + self.nbytes:]
        ok = bool((head == SENTINEL).all()) and bool((tail == SENTINEL).all())
        assert ok, f"{what}: a kernel wrote outside its output buffer"


def need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def oracle_pack_vals(W: np.ndarray, G: int, K: int, val_dtype):
    """Oracle pack; returns (vals in the storage dtype as exact fp32 values,
    idx, and the storage bit pattern for bit-exact comparison)."""
    v32, idx = oracle.pack(W, G, K)
    if val_dtype == torch.bfloat16:
        bits = oracle.bf16_rne(v32)
        return oracle.bf16_bits_to_f32(bits), idx, bits
    return v32, idx, v32.view(np.uint32)


def gpu_bits(vals: torch.Tensor):
    if vals.dtype == torch.bfloat16:
        return bits_u16(vals)
    return vals.detach().cpu().numpy().view(np.uint32)


def x_as_f32(X: torch.Tensor) -> np.ndarray:
    return X.detach().float().cpu().numpy()


def epilogue_terms(Yabs, scale, bias, res):
    S = Yabs.copy()
    if scale is not None:
        S = S * np.abs(scale)[None, :]
    if bias is not None:
        S = S + np.abs(bias)[None, :]
    if res is not None:
        S = S + np.abs(res)
    return S


def tol_for(y_dtype, x_dtype):
    return TOL["f32"] if (x_dtype == torch.float32 and y_dtype == torch.float32) else TOL["bf16"]


def rand_epilogue(O, N, y_dtype, seed, scale=True, bias=True, residual=False, relu=False):
    rng = np.random.default_rng(seed)
    s = (0.5 + rng.random(O)).astype(np.float32) if scale else None
    b = (0.1 * rng.standard_normal(O)).astype(np.float32) if bias else None
    r = None
    r_t = None
    if residual:
        r_t = torch.from_numpy(rng.standard_normal((N, O)).astype(np.float32)).to(y_dtype)
        r = r_t.float().numpy()
    return s, b, r, r_t, relu
