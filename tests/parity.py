"""Comparison rules for GPU results against the CPU oracle.

Floating-point outputs pass two checks (tolerance `tol`: 1e-5 for fp32,
1e-2 for bf16-in / fp32-accumulate):
  1. max |Y_gpu - Y_ref| / max |Y_ref|  <= tol     (per output tensor)
  2. |Y_gpu - Y_ref| <= tol * S + tiny per element, where S is the sum of the
     magnitudes of every term that entered that output (products, scaled,
     plus |bias| and |residual|) -- the scale of any rounding error.
Integer / index outputs and packed values must be bit-identical.
"""
import numpy as np
import torch

TOL = {"f32": 1e-5, "bf16": 1e-2}


def to_np_f32(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy()


def bits_u16(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)


def check_close(got: np.ndarray, ref: np.ndarray, scale_terms: np.ndarray, tol: float, what: str):
    got = np.asarray(got, np.float64).reshape(ref.shape)
    assert np.all(np.isfinite(got)), f"{what}: non-finite GPU output"
    err = np.abs(got - ref)
    denom = max(np.abs(ref).max(), 1e-30)
    rel = err.max() / denom
    assert rel <= tol, f"{what}: max|err|/max|ref| = {rel:.3e} > {tol}"
    bound = tol * np.asarray(scale_terms).reshape(ref.shape) + 1e-30
    bad = err > bound
    assert not bad.any(), (f"{what}: {int(bad.sum())} elements exceed tol*sum|terms|; "
                           f"worst ratio {(err / bound).max():.3e}")
    return rel
