"""CPU oracle for the CCI-sparse forward path -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s cpu_baseline
leg may import this package.  It imports nothing from the HIP library's
package, and the HIP library imports nothing from here.

Every arithmetic step lives in ``cci_oracle.c`` (plain C, double precision);
this module only marshals numpy arrays.  Each wrapper names the passage of
the paper (Yu et al., arXiv:1910.11971) that its C function follows.

Parity status of each function (what pins it, see ``tests/test_oracle.py``):
  pack          brute-force top-K over all subsets; Sec. 3.3 worked example;
                Fig. 1 counts; Eq. 1 Monte-Carlo; K=G identity; K=1 argmax
  unpack        round trip with pack; hand example (tests/golden)
  spmm_rows     numpy float64 matmul of the masked matrix; K=G plain product;
                one-hot input; exact small-integer hand example (tests/golden)
  dense_rows    numpy float64 matmul
  conv2d_nhwc   torch.nn.functional.conv2d (float64, CPU); 1x1 conv == FC;
                im2col + spmm
  im2col_nhwc   torch.nn.functional.unfold (float64, CPU), reordered
  bf16_rne      torch float32 -> bfloat16 conversion; hand-built tie cases
  maxpool2d     torch.nn.functional.max_pool2d (CPU)
  avgpool       numpy mean
  eq1_pd        exact rationals evaluated by hand (tests/golden/eq1_values.txt)
"""
from __future__ import annotations

import ctypes
import os
from fractions import Fraction
from math import comb

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None

_f32p = ctypes.POINTER(ctypes.c_float)
_f64p = ctypes.POINTER(ctypes.c_double)
_u8p = ctypes.POINTER(ctypes.c_uint8)
_u16p = ctypes.POINTER(ctypes.c_uint16)
_i64p = ctypes.POINTER(ctypes.c_int64)
_i64 = ctypes.c_int64
_i32 = ctypes.c_int32


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        from . import build as _build  # noqa: WPS433 (builds the checker only)
        _build.build()
    lib = ctypes.CDLL(_LIB_PATH)
    lib.oracle_pack.argtypes = [_f32p, _i64, _i64, _i32, _i32, _f32p, _u8p]
    lib.oracle_unpack.argtypes = [_f32p, _u8p, _i64, _i64, _i32, _i32, _f32p]
    lib.oracle_spmm_rows.argtypes = [
        _f32p, _i64, _i64, _f32p, _u8p, _i64, _i32, _i32,
        _f32p, _f32p, _f32p, _i32, _i64p, _i64, _f64p, _f64p]
    lib.oracle_dense_rows.argtypes = [
        _f32p, _i64, _i64, _f32p, _i64, _f32p, _f32p, _f32p, _i32,
        _i64p, _i64, _f64p]
    lib.oracle_conv2d_nhwc_rows.argtypes = [
        _f32p, _i64, _i64, _i64, _i64, _f32p, _i64, _i32, _i32, _i32, _i32,
        _i32, _i32, _f32p, _f32p, _f32p, _i32, _i64p, _i64, _f64p, _f64p]
    lib.oracle_im2col_nhwc.argtypes = [
        _f32p, _i64, _i64, _i64, _i64, _i32, _i32, _i32, _i32, _i32, _i32,
        _f32p]
    lib.oracle_bf16_rne.argtypes = [ctypes.c_float]
    lib.oracle_bf16_rne.restype = ctypes.c_uint16
    lib.oracle_bf16_rne_array.argtypes = [_f32p, _u16p, _i64]
    lib.oracle_maxpool2d_nhwc.argtypes = [
        _f32p, _i64, _i64, _i64, _i64, _i32, _i32, _i32, _f32p]
    lib.oracle_global_avgpool_nhwc.argtypes = [
        _f32p, _i64, _i64, _i64, _i64, _f64p]
    lib.oracle_bbs_pack.argtypes = [_f32p, _i64, _i64, _i32, _i32, _f32p, _u8p]
    lib.oracle_bbs_unpack.argtypes = [_f32p, _u8p, _i64, _i64, _i32, _i32, _f32p]
    lib.oracle_bbs_spmm_rows.argtypes = [
        _f32p, _i64, _i64, _f32p, _u8p, _i64, _i32, _i32,
        _f32p, _f32p, _f32p, _i32, _i64p, _i64, _f64p, _f64p]
    lib.oracle_td_schedule.argtypes = [_i64, _i64, _i32, _i32, ctypes.POINTER(_i32), ctypes.POINTER(ctypes.c_double)]
    lib.oracle_td_mask.argtypes = [_f32p, _i64, _i64, _i32, _i32, ctypes.POINTER(ctypes.c_uint32), ctypes.c_double,
                                   _f32p, _u8p]
    lib.oracle_grad_packed.argtypes = [_f32p, _f32p, _i64, _i64, _u8p, _i64, _i32, _i32, _f64p]
    lib.oracle_index_width.argtypes = [_i32]
    lib.oracle_index_width.restype = _i32
    lib.oracle_index_bits.argtypes = [_u8p, _i64, _i32, ctypes.POINTER(ctypes.c_uint32)]
    lib.oracle_index_unbits.argtypes = [ctypes.POINTER(ctypes.c_uint32), _i64, _i32, _u8p]
    lib.oracle_num_threads.restype = ctypes.c_int
    lib.oracle_set_num_threads.argtypes = [ctypes.c_int]
    lib.oracle_set_num_threads.restype = None
    for fn in ("oracle_pack", "oracle_unpack", "oracle_spmm_rows",
               "oracle_dense_rows", "oracle_conv2d_nhwc_rows",
               "oracle_im2col_nhwc", "oracle_maxpool2d_nhwc",
               "oracle_global_avgpool_nhwc", "oracle_bbs_pack", "oracle_bbs_unpack",
               "oracle_bbs_spmm_rows", "oracle_td_schedule", "oracle_td_mask", "oracle_grad_packed",
               "oracle_index_bits", "oracle_index_unbits"):
        getattr(lib, fn).restype = ctypes.c_int
    _lib = lib
    return lib


def _p(a: np.ndarray | None, ptype):
    if a is None:
        return ctypes.cast(None, ptype)
    return a.ctypes.data_as(ptype)


def _f32(a):
    return None if a is None else np.ascontiguousarray(a, dtype=np.float32)


def _check(rc: int, what: str):
    if rc != 0:
        raise ValueError(f"oracle {what}: invalid arguments (rc={rc})")


def num_threads() -> int:
    return int(_load().oracle_num_threads())


def set_num_threads(n: int) -> None:
    """Threads of the oracle's later parallel loops (timing only)."""
    _load().oracle_set_num_threads(int(n))


def pack(W: np.ndarray, G: int, K: int):
    """Per-group top-K by |w| (Sec. 5.1; Sec. 3.1, Fig. 1).

    W: fp32 [O, C].  Returns (vals fp32 [O/G, K, C], idx uint8 [O/G, K, C]);
    kept rows in ascending r; ties between equal |w| go to the lower r.
    """
    W = _f32(W)
    O, C = W.shape
    if G < 1 or O % G:
        raise ValueError("O must be a positive multiple of G")
    vals = np.empty((O // G, K, C), np.float32)
    idx = np.empty((O // G, K, C), np.uint8)
    _check(_load().oracle_pack(_p(W, _f32p), O, C, G, K, _p(vals, _f32p),
                               _p(idx, _u8p)), "pack")
    return vals, idx


def unpack(vals: np.ndarray, idx: np.ndarray, G: int) -> np.ndarray:
    """Dense masked matrix [O, C] described by a packed pair (Sec. 3.1)."""
    vals = _f32(vals)
    idx = np.ascontiguousarray(idx, dtype=np.uint8)
    ng, K, C = vals.shape
    O = ng * G
    Wd = np.empty((O, C), np.float32)
    _check(_load().oracle_unpack(_p(vals, _f32p), _p(idx, _u8p), O, C, G, K,
                                 _p(Wd, _f32p)), "unpack")
    return Wd


def spmm_rows(X, vals, idx, G, *, scale=None, bias=None, residual=None,
              relu=False, rows=None, want_abs=False):
    """Alg. 1 (Sec. 3.2) generalised to K slots, in double, plus epilogue.

    X fp32 [N, C]; vals fp32 [O/G, K, C] (pass bf16 weights as their exact
    fp32 values); idx uint8.  Returns Y float64 [len(rows) or N, O] (and the
    per-output sum of |products| when want_abs).
    """
    X = _f32(X)
    vals = _f32(vals)
    idx = np.ascontiguousarray(idx, dtype=np.uint8)
    N, C = X.shape
    ng, K, C2 = vals.shape
    if C2 != C or idx.shape != vals.shape:
        raise ValueError("shape mismatch")
    O = ng * G
    rows_a = None if rows is None else np.ascontiguousarray(rows, np.int64)
    nrows = N if rows_a is None else rows_a.shape[0]
    Y = np.empty((nrows, O), np.float64)
    Yabs = np.empty((nrows, O), np.float64) if want_abs else None
    _check(_load().oracle_spmm_rows(
        _p(X, _f32p), N, C, _p(vals, _f32p), _p(idx, _u8p), O, G, K,
        _p(_f32(scale), _f32p), _p(_f32(bias), _f32p),
        _p(_f32(residual), _f32p), int(bool(relu)), _p(rows_a, _i64p), nrows,
        _p(Y, _f64p), _p(Yabs, _f64p)), "spmm_rows")
    return (Y, Yabs) if want_abs else Y


def dense_rows(X, Wd, *, scale=None, bias=None, residual=None, relu=False,
               rows=None):
    """Alg. 0 (Sec. 3.2): dense product with an unpacked [O, C] matrix."""
    X = _f32(X)
    Wd = _f32(Wd)
    N, C = X.shape
    O = Wd.shape[0]
    rows_a = None if rows is None else np.ascontiguousarray(rows, np.int64)
    nrows = N if rows_a is None else rows_a.shape[0]
    Y = np.empty((nrows, O), np.float64)
    _check(_load().oracle_dense_rows(
        _p(X, _f32p), N, C, _p(Wd, _f32p), O, _p(_f32(scale), _f32p),
        _p(_f32(bias), _f32p), _p(_f32(residual), _f32p), int(bool(relu)),
        _p(rows_a, _i64p), nrows, _p(Y, _f64p)), "dense_rows")
    return Y


def conv_out_hw(H, W, KH, KW, stride, pad):
    sh, sw = stride
    ph, pw = pad
    return (H + 2 * ph - KH) // sh + 1, (W + 2 * pw - KW) // sw + 1


def conv2d_nhwc(X, Wd, stride=(1, 1), pad=(0, 0), *, scale=None, bias=None,
                residual=None, relu=False, pixels=None, want_abs=False):
    """Direct convolution from the definition (Sec. 3.2 lowers it to GEMM).

    X fp32 NHWC [B, H, W, Cin]; Wd fp32 [O, KH, KW, Cin] (dense / masked).
    Returns Y float64 [npix, O] over output pixels p = (b*Ho+oh)*Wo+ow.
    """
    X = _f32(X)
    Wd = _f32(Wd)
    B, H, W, Cin = X.shape
    O, KH, KW, Cin2 = Wd.shape
    if Cin2 != Cin:
        raise ValueError("Cin mismatch")
    Ho, Wo = conv_out_hw(H, W, KH, KW, stride, pad)
    pix = None if pixels is None else np.ascontiguousarray(pixels, np.int64)
    npix = B * Ho * Wo if pix is None else pix.shape[0]
    Y = np.empty((npix, O), np.float64)
    Yabs = np.empty((npix, O), np.float64) if want_abs else None
    _check(_load().oracle_conv2d_nhwc_rows(
        _p(X, _f32p), B, H, W, Cin, _p(Wd, _f32p), O, KH, KW, stride[0],
        stride[1], pad[0], pad[1], _p(_f32(scale), _f32p),
        _p(_f32(bias), _f32p), _p(_f32(residual), _f32p), int(bool(relu)),
        _p(pix, _i64p), npix, _p(Y, _f64p), _p(Yabs, _f64p)), "conv2d_nhwc")
    return (Y, Yabs) if want_abs else Y


def im2col_nhwc(X, KH, KW, stride=(1, 1), pad=(0, 0)):
    """Explicit im2col, columns in (kh, kw, cin) order."""
    X = _f32(X)
    B, H, W, Cin = X.shape
    Ho, Wo = conv_out_hw(H, W, KH, KW, stride, pad)
    A = np.empty((B * Ho * Wo, KH * KW * Cin), np.float32)
    _check(_load().oracle_im2col_nhwc(
        _p(X, _f32p), B, H, W, Cin, KH, KW, stride[0], stride[1], pad[0],
        pad[1], _p(A, _f32p)), "im2col_nhwc")
    return A


def bf16_rne(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns (uint16), round to nearest even."""
    x = _f32(x)
    out = np.empty(x.shape, np.uint16)
    _load().oracle_bf16_rne_array(_p(x, _f32p), _p(out, _u16p), x.size)
    return out


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to fp32 (bits move up 16 places)."""
    return (np.asarray(bits, np.uint16).astype(np.uint32) << 16).view(np.float32)


def maxpool2d_nhwc(X, k, s, p):
    X = _f32(X)
    B, H, W, C = X.shape
    Ho, Wo = (H + 2 * p - k) // s + 1, (W + 2 * p - k) // s + 1
    Y = np.empty((B, Ho, Wo, C), np.float32)
    _check(_load().oracle_maxpool2d_nhwc(_p(X, _f32p), B, H, W, C, k, s, p,
                                         _p(Y, _f32p)), "maxpool2d_nhwc")
    return Y


def global_avgpool_nhwc(X):
    X = _f32(X)
    B, H, W, C = X.shape
    Y = np.empty((B, C), np.float64)
    _check(_load().oracle_global_avgpool_nhwc(_p(X, _f32p), B, H, W, C,
                                              _p(Y, _f64p)), "avgpool")
    return Y


def eq1_pd(G: int, Ps: Fraction) -> Fraction:
    """Paper Sec. 4, Eq. 1: probability that a nonzero weight finds no slot.

    Each weight is nonzero independently with probability 1 - Ps; a group of
    G has s = G (1 - Ps) slots; with i ~ Binomial(G, 1 - Ps) nonzeros a group
    discards max(i - s, 0) of them.  P_d = sum_{i=1}^{G} 1(i > s) (i - s)
    B(i; G, 1 - Ps) / s, evaluated exactly in rationals.
    """
    Ps = Fraction(Ps)
    q = 1 - Ps
    s = G * q
    if s.denominator != 1 or s < 1:
        raise ValueError("s = G(1-Ps) must be a positive integer")
    s = int(s)
    total = Fraction(0)
    for i in range(1, G + 1):
        if i > s:
            total += (i - s) * comb(G, i) * q ** i * Ps ** (G - i)
    return total / s


# ------------------------------------------------------- balanced sparsity --

def bbs_pack(W: np.ndarray, G: int, K: int):
    """Balanced-sparsity projection (Sec. 2.4, Sec. 3.3, Fig. 2b): per row,
    per group of G contiguous inputs, keep the K largest |w| (ties: lower
    position), ascending.  W fp32 [O, C], C % G == 0.  Returns (vals fp32
    [O, C/G, K], idx uint8 [O, C/G, K])."""
    W = _f32(W)
    O, C = W.shape
    if G < 1 or C % G:
        raise ValueError("C must be a multiple of G")
    vals = np.empty((O, C // G, K), np.float32)
    idx = np.empty((O, C // G, K), np.uint8)
    _check(_load().oracle_bbs_pack(_p(W, _f32p), O, C, G, K, _p(vals, _f32p), _p(idx, _u8p)), "bbs_pack")
    return vals, idx


def bbs_unpack(vals: np.ndarray, idx: np.ndarray, G: int) -> np.ndarray:
    """The dense masked [O, C] matrix of a balanced-sparse packing."""
    vals = _f32(vals)
    idx = np.ascontiguousarray(idx, np.uint8)
    O, ng, K = vals.shape
    Wd = np.empty((O, ng * G), np.float32)
    _check(_load().oracle_bbs_unpack(_p(vals, _f32p), _p(idx, _u8p), O, ng * G, G, K, _p(Wd, _f32p)), "bbs_unpack")
    return Wd


def bbs_spmm_rows(X, vals, idx, G, *, scale=None, bias=None, residual=None, relu=False, rows=None,
                  want_abs=False):
    """Balanced-sparse product (Sec. 3.3, Fig. 2b) in double precision:
    Y[n][o] = epilogue(sum_j sum_k vals[o][j][k] * X[n][jG + idx[o][j][k]])."""
    X = _f32(X)
    vals = _f32(vals)
    idx = np.ascontiguousarray(idx, np.uint8)
    N, C = X.shape
    O, ng, K = vals.shape
    if ng * G != C:
        raise ValueError("packed groups do not match X")
    r = None if rows is None else np.ascontiguousarray(rows, np.int64)
    nrows = N if r is None else r.shape[0]
    Y = np.empty((nrows, O), np.float64)
    Yabs = np.empty((nrows, O), np.float64) if want_abs else None
    _check(_load().oracle_bbs_spmm_rows(
        _p(X, _f32p), N, C, _p(vals, _f32p), _p(idx, _u8p), O, G, K, _p(_f32(scale), _f32p),
        _p(_f32(bias), _f32p), _p(_f32(residual), _f32p), int(bool(relu)), _p(r, _i64p), nrows,
        _p(Y, _f64p), _p(Yabs, _f64p)), "bbs_spmm_rows")
    return (Y, Yabs) if want_abs else Y


# ------------------------------------------------ improved targeted dropout --

def td_schedule(step: int, total: int, G: int, K: int):
    """(n_target candidates per group, candidate dropout rate) at `step` of
    `total` (Sec. 5.1, Sec. 6)."""
    n = _i32()
    p = ctypes.c_double()
    _check(_load().oracle_td_schedule(step, total, G, K, ctypes.byref(n), ctypes.byref(p)), "td_schedule")
    return n.value, p.value


def td_mask(W: np.ndarray, G: int, n_target: int, bits: np.ndarray, drop_rate: float):
    """Candidate dropout of one step: (W_eff fp32 [O, C], keep uint8 [O, C])."""
    W = _f32(W)
    O, C = W.shape
    bits = np.ascontiguousarray(bits, np.uint32)
    if bits.shape != (O, C):
        raise ValueError("bits must be uint32 [O, C]")
    We = np.empty((O, C), np.float32)
    keep = np.empty((O, C), np.uint8)
    _check(_load().oracle_td_mask(_p(W, _f32p), O, C, G, n_target, bits.ctypes.data_as(ctypes.POINTER(ctypes.c_uint32)),
                                  float(drop_rate), _p(We, _f32p), _p(keep, _u8p)), "td_mask")
    return We, keep


def grad_packed(dY, X, idx, G):
    """dL/dvals [O/G, K, C] of Y = X W_hat^T for dY [N, O], X [N, C] (double)."""
    dY = _f32(dY)
    X = _f32(X)
    idx = np.ascontiguousarray(idx, np.uint8)
    N, O = dY.shape
    ng, K, C = idx.shape
    if X.shape != (N, C) or ng * G != O:
        raise ValueError("shape mismatch")
    out = np.empty((ng, K, C), np.float64)
    _check(_load().oracle_grad_packed(_p(dY, _f32p), _p(X, _f32p), N, C, _p(idx, _u8p), O, G, K, _p(out, _f64p)),
           "grad_packed")
    return out


# ------------------------------------------------------ log2(G)-bit indices --

def index_width(G: int) -> int:
    """Bits of a plain intra-group index (Sec. 3.1): ceil(log2 G), at least 1."""
    b = int(_load().oracle_index_width(G))
    if b < 0:
        raise ValueError("G outside [1, 256]")
    return b


def index_bits(idx: np.ndarray, b: int) -> np.ndarray:
    """The index array as a little-endian b-bit stream (uint32 words)."""
    idx = np.ascontiguousarray(idx, np.uint8).reshape(-1)
    words = np.empty(((idx.size * b + 31) // 32,), np.uint32)
    _check(_load().oracle_index_bits(_p(idx, _u8p), idx.size, b,
                                     words.ctypes.data_as(ctypes.POINTER(ctypes.c_uint32))), "index_bits")
    return words


def index_unbits(words: np.ndarray, n: int, b: int) -> np.ndarray:
    words = np.ascontiguousarray(words, np.uint32)
    if words.size < (n * b + 31) // 32:
        raise ValueError("stream too short")
    idx = np.empty((n,), np.uint8)
    _check(_load().oracle_index_unbits(words.ctypes.data_as(ctypes.POINTER(ctypes.c_uint32)), n, b, _p(idx, _u8p)),
           "index_unbits")
    return idx
