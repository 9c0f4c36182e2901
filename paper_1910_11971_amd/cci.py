"""Python binding of the C ABI in include/cci.h (argument marshalling only).

Every function takes and returns torch tensors on a HIP device; the work is
enqueued on the current torch stream of that device and runs in the HIP
kernels of ``libcci.so``.  There is no fallback: if the library is missing,
importing this module raises.
"""
from __future__ import annotations

import ctypes
import os
import re

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libcci.so")
HEADER_PATH = os.path.join(os.path.dirname(_HERE), "include", "cci.h")

OK, EINVAL, EUNSUPPORTED, EALIGN, EHIP = 0, 1, 2, 3, 4
F32, BF16 = 0, 1
(ALGO_AUTO, ALGO_SPARSE_MAC, ALGO_DENSE_TILE_MFMA, ALGO_WIDE_TILE_MFMA, ALGO_NARROW_MFMA, ALGO_RESIDENT_MFMA,
 ALGO_FEW_ROWS_MFMA, ALGO_TAP_TILE_MFMA, ALGO_STREAM_TILE_MFMA, ALGO_SPLIT_K_MFMA) = range(10)
ALGOS = {"auto": ALGO_AUTO, "sparse_mac": ALGO_SPARSE_MAC, "dense_tile_mfma": ALGO_DENSE_TILE_MFMA,
         "wide_tile_mfma": ALGO_WIDE_TILE_MFMA, "narrow_mfma": ALGO_NARROW_MFMA,
         "resident_mfma": ALGO_RESIDENT_MFMA, "few_rows_mfma": ALGO_FEW_ROWS_MFMA,
         "tap_tile_mfma": ALGO_TAP_TILE_MFMA, "stream_tile_mfma": ALGO_STREAM_TILE_MFMA,
         "split_k_mfma": ALGO_SPLIT_K_MFMA}


class CCIError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"status {status}: {msg}")
        self.status = status


class Epilogue(ctypes.Structure):
    _fields_ = [("scale", ctypes.c_void_p), ("bias", ctypes.c_void_p),
                ("residual", ctypes.c_void_p), ("relu", ctypes.c_int32)]


if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_1910_11971_amd.build`")

# torch is imported first so that its HIP runtime (same soname) is the one
# libcci.so binds to: one runtime per process.
_lib = ctypes.CDLL(LIB_PATH)
_vp, _i64, _i32, _sz = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_size_t
_lib.cci_packed_sizes.argtypes = [_i64, _i64, _i32, _i32, ctypes.c_int, ctypes.POINTER(_sz), ctypes.POINTER(_sz)]
_lib.cci_pack.argtypes = [_vp, _i64, _i64, _i32, _i32, _vp, ctypes.c_int, _vp, _vp]
_SPMM = [_vp, ctypes.c_int, _i64, _i64, _vp, ctypes.c_int, _vp, _i64, _i32, _i32, ctypes.POINTER(Epilogue), _vp,
         ctypes.c_int]
_CONV = [_vp, ctypes.c_int, _i64, _i64, _i64, _i64, _i32, _i32, _i32, _i32, _i32, _i32, _vp, ctypes.c_int, _vp,
         _i64, _i32, _i32, ctypes.POINTER(Epilogue), _vp, ctypes.c_int]
_lib.cci_spmm.argtypes = _SPMM + [_vp]
_lib.cci_spmm_algo.argtypes = _SPMM + [ctypes.c_int, _vp]
_lib.cci_conv_im2col.argtypes = _CONV + [_vp]
_lib.cci_conv_im2col_algo.argtypes = _CONV + [ctypes.c_int, _vp]
_lib.cci_bbs_packed_sizes.argtypes = [_i64, _i64, _i32, _i32, ctypes.c_int, ctypes.POINTER(_sz), ctypes.POINTER(_sz)]
_lib.cci_bbs_pack.argtypes = [_vp, _i64, _i64, _i32, _i32, _vp, ctypes.c_int, _vp, _vp]
_lib.cci_2of4_sizes.argtypes = [_i64, _i64, ctypes.POINTER(_sz), ctypes.POINTER(_sz)]
_lib.cci_bbs_to_2of4.argtypes = [_vp, ctypes.c_int, _vp, _i64, _i64, _i32, _i32, _vp, _vp, _vp]
_lib.cci_to_2of4_transposed.argtypes = [_vp, ctypes.c_int, _vp, _i64, _i64, _i32, _i32, _vp, _vp, _vp]
_lib.cci_spmm_2of4.argtypes = [_vp, ctypes.c_int, _i64, _i64, _vp, _vp, _i64, ctypes.POINTER(Epilogue), _vp,
                               ctypes.c_int, _vp]
_lib.cci_td_schedule.argtypes = [_i64, _i64, _i32, _i32, ctypes.POINTER(_i32), ctypes.POINTER(ctypes.c_double)]
_lib.cci_td_mask.argtypes = [_vp, _i64, _i64, _i32, _i32, _vp, ctypes.c_double, _vp, ctypes.c_int, _vp, _vp]
_lib.cci_grad_packed.argtypes = [_vp, _vp, ctypes.c_int, _i64, _i64, _vp, _i64, _i32, _i32, _vp, _vp]
_lib.cci_index_width.argtypes = [_i32]
_lib.cci_index_width.restype = _i32
_lib.cci_index_stream_bytes.argtypes = [_i64, _i32, ctypes.POINTER(_sz)]
_lib.cci_index_bits.argtypes = [_vp, _i64, _i32, _vp, _vp]
_lib.cci_spmm_bits.argtypes = [_vp, ctypes.c_int, _i64, _i64, _vp, ctypes.c_int, _vp, _i32, _i64, _i32, _i32,
                               ctypes.POINTER(Epilogue), _vp, ctypes.c_int, _vp]
_lib.cci_auto_algo.argtypes = [ctypes.c_int, ctypes.c_int, _i64, _i64, _i64, _i64, _i32, _i32]
_lib.cci_auto_algo.restype = ctypes.c_int
_lib.cci_maxpool2d_nhwc.argtypes = [_vp, ctypes.c_int, _i64, _i64, _i64, _i64, _i32, _i32, _i32, _vp, _vp]
_lib.cci_global_avgpool_nhwc.argtypes = [_vp, ctypes.c_int, _i64, _i64, _i64, _i64, _vp, ctypes.c_int, _vp]
_lib.cci_status_str.argtypes = [ctypes.c_int]
_lib.cci_status_str.restype = ctypes.c_char_p
_lib.cci_last_error.restype = ctypes.c_char_p
_lib.cci_version.restype = ctypes.c_int32
for _fn in ("cci_packed_sizes", "cci_pack", "cci_spmm", "cci_spmm_algo", "cci_conv_im2col",
            "cci_conv_im2col_algo", "cci_maxpool2d_nhwc", "cci_global_avgpool_nhwc", "cci_bbs_packed_sizes",
            "cci_bbs_pack", "cci_2of4_sizes", "cci_bbs_to_2of4", "cci_to_2of4_transposed", "cci_spmm_2of4",
            "cci_td_schedule", "cci_td_mask", "cci_grad_packed", "cci_index_stream_bytes", "cci_index_bits",
            "cci_spmm_bits"):
    getattr(_lib, _fn).restype = ctypes.c_int


def raw():
    """The loaded ctypes library (for ABI-level tests)."""
    return _lib


def header_functions() -> list[str]:
    """Names of the functions include/cci.h declares."""
    with open(HEADER_PATH) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(cci_[a-z0-9_]+)\s*\(", text)))


def _check(status: int):
    if status != OK:
        raise CCIError(status, _lib.cci_last_error().decode() or _lib.cci_status_str(status).decode())


def _code(dt: torch.dtype) -> int:
    if dt == torch.float32:
        return F32
    if dt == torch.bfloat16:
        return BF16
    raise TypeError(f"unsupported dtype {dt}")


def _ptr(t: torch.Tensor | None):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _dev(t: torch.Tensor) -> torch.Tensor:
    if not t.is_cuda:
        raise ValueError("tensor must be on a HIP device")
    if not t.is_contiguous():
        raise ValueError("tensor must be contiguous")
    return t


def _stream(t: torch.Tensor):
    return ctypes.c_void_p(torch.cuda.current_stream(t.device).cuda_stream)


def _algo(algo) -> int:
    return ALGOS[algo] if isinstance(algo, str) else int(algo)


def version() -> int:
    return int(_lib.cci_version())


def packed_sizes(O: int, C: int, G: int, K: int, val_dtype=torch.bfloat16):
    vb, ib = _sz(), _sz()
    _check(_lib.cci_packed_sizes(O, C, G, K, _code(val_dtype), ctypes.byref(vb), ctypes.byref(ib)))
    return vb.value, ib.value


def pack(W: torch.Tensor, G: int, K: int, val_dtype=torch.bfloat16, out=None):
    """cci_pack: W fp32 [O, C] (conv: [O, KH, KW, Cin]) -> (vals [O/G, K, C], idx uint8).

    `out=(vals, idx)` writes into caller tensors of exactly that shape and dtype."""
    _dev(W)
    if W.dtype != torch.float32:
        raise TypeError("W must be float32")
    O = W.shape[0]
    C = W.numel() // max(O, 1)
    if O % G:
        raise ValueError("O must be a multiple of G")
    if out is None:
        vals = torch.empty((O // G, K, C), dtype=val_dtype, device=W.device)
        idx = torch.empty((O // G, K, C), dtype=torch.uint8, device=W.device)
    else:
        vals, idx = out
        _dev(vals), _dev(idx)
        if (tuple(vals.shape) != (O // G, K, C) or tuple(idx.shape) != (O // G, K, C)
                or vals.dtype != val_dtype or idx.dtype != torch.uint8
                or not vals.is_contiguous() or not idx.is_contiguous()):
            raise ValueError("out must be contiguous (vals, idx) of shape [O/G, K, C] with the packed dtypes")
    _check(_lib.cci_pack(_ptr(W), O, C, G, K, _ptr(vals), _code(val_dtype), _ptr(idx), _stream(W)))
    return vals, idx


def _epilogue(scale, bias, residual, relu, O, y_shape, y_dtype, device):
    """Marshal the fused epilogue after checking what the kernels will read:
    scale / bias fp32 [O], residual of Y's shape and dtype, all contiguous
    on Y's device."""
    for name, t in (("scale", scale), ("bias", bias)):
        if t is not None:
            _dev(t)
            if t.dtype != torch.float32 or t.numel() != O or t.device != device:
                raise ValueError(f"{name} must be a contiguous float32 tensor of {O} elements on {device}")
    if residual is not None:
        _dev(residual)
        if tuple(residual.shape) != tuple(y_shape) or residual.dtype != y_dtype or residual.device != device:
            raise ValueError(f"residual must be a contiguous {y_dtype} tensor of shape {tuple(y_shape)} on {device}")
    return Epilogue(_ptr(scale), _ptr(bias), _ptr(residual), int(bool(relu)))


def _out(out, shape, dtype, device):
    if out is None:
        return torch.empty(shape, dtype=dtype, device=device)
    _dev(out)
    if tuple(out.shape) != tuple(shape) or out.dtype != dtype or out.device != device:
        raise ValueError(f"out must be a contiguous {dtype} tensor of shape {tuple(shape)} on {device}")
    return out


def spmm(X: torch.Tensor, vals: torch.Tensor, idx: torch.Tensor, G: int, *, scale=None, bias=None,
         residual=None, relu=False, out_dtype=None, algo="auto", out=None) -> torch.Tensor:
    """cci_spmm (cci_spmm_algo when `algo` pins a kernel family):
    Y [N, O] = epilogue(X [N, C] . W_hat^T) from packed (vals, idx)."""
    _dev(X), _dev(vals), _dev(idx)
    N, C = X.shape
    ng, K, C2 = vals.shape
    if C2 != C or tuple(idx.shape) != tuple(vals.shape) or idx.dtype != torch.uint8:
        raise ValueError("shape mismatch between X and packed weights")
    if vals.device != X.device or idx.device != X.device:
        raise ValueError("X and the packed weights must be on one device")
    O = ng * G
    Y = _out(out, (N, O), out_dtype or X.dtype, X.device)
    ep = _epilogue(scale, bias, residual, relu, O, Y.shape, Y.dtype, X.device)
    args = (_ptr(X), _code(X.dtype), N, C, _ptr(vals), _code(vals.dtype), _ptr(idx), O, G, K, ctypes.byref(ep),
            _ptr(Y), _code(Y.dtype))
    a = _algo(algo)
    _check(_lib.cci_spmm(*args, _stream(X)) if a == ALGO_AUTO else _lib.cci_spmm_algo(*args, a, _stream(X)))
    return Y


def conv_out_hw(H, W, KH, KW, stride, pad):
    return (H + 2 * pad[0] - KH) // stride[0] + 1, (W + 2 * pad[1] - KW) // stride[1] + 1


def conv_im2col(X: torch.Tensor, vals: torch.Tensor, idx: torch.Tensor, G: int, KH: int, KW: int,
                stride=(1, 1), pad=(0, 0), *, scale=None, bias=None, residual=None, relu=False,
                out_dtype=None, algo="auto", out=None) -> torch.Tensor:
    """cci_conv_im2col (cci_conv_im2col_algo when `algo` pins a kernel
    family): NHWC X [B, H, W, Cin] -> NHWC Y [B, Ho, Wo, O]."""
    _dev(X), _dev(vals), _dev(idx)
    B, H, W, Cin = X.shape
    ng, K, C = vals.shape
    if C != KH * KW * Cin or tuple(idx.shape) != tuple(vals.shape) or idx.dtype != torch.uint8:
        raise ValueError("packed weights do not match KH*KW*Cin")
    if vals.device != X.device or idx.device != X.device:
        raise ValueError("X and the packed weights must be on one device")
    O = ng * G
    Ho, Wo = conv_out_hw(H, W, KH, KW, stride, pad)
    Y = _out(out, (B, Ho, Wo, O), out_dtype or X.dtype, X.device)
    ep = _epilogue(scale, bias, residual, relu, O, Y.shape, Y.dtype, X.device)
    args = (_ptr(X), _code(X.dtype), B, H, W, Cin, KH, KW, stride[0], stride[1], pad[0], pad[1], _ptr(vals),
            _code(vals.dtype), _ptr(idx), O, G, K, ctypes.byref(ep), _ptr(Y), _code(Y.dtype))
    a = _algo(algo)
    _check(_lib.cci_conv_im2col(*args, _stream(X)) if a == ALGO_AUTO
           else _lib.cci_conv_im2col_algo(*args, a, _stream(X)))
    return Y


def auto_algo(x_dtype, val_dtype, N, C, cin, O, G, K) -> str:
    code = _lib.cci_auto_algo(_code(x_dtype), _code(val_dtype), N, C, cin, O, G, K)
    return {v: k for k, v in ALGOS.items()}[code]


def maxpool2d_nhwc(X: torch.Tensor, k: int, s: int, p: int) -> torch.Tensor:
    _dev(X)
    B, H, W, C = X.shape
    Ho, Wo = (H + 2 * p - k) // s + 1, (W + 2 * p - k) // s + 1
    Y = torch.empty((B, Ho, Wo, C), dtype=X.dtype, device=X.device)
    _check(_lib.cci_maxpool2d_nhwc(_ptr(X), _code(X.dtype), B, H, W, C, k, s, p, _ptr(Y), _stream(X)))
    return Y


def global_avgpool_nhwc(X: torch.Tensor, out_dtype=None) -> torch.Tensor:
    _dev(X)
    B, H, W, C = X.shape
    Y = torch.empty((B, C), dtype=out_dtype or X.dtype, device=X.device)
    _check(_lib.cci_global_avgpool_nhwc(_ptr(X), _code(X.dtype), B, H, W, C, _ptr(Y), _code(Y.dtype),
                                        _stream(X)))
    return Y


# ------------------------------------------------------- balanced sparsity --

def bbs_pack(W: torch.Tensor, G: int, K: int, val_dtype=torch.bfloat16, out=None):
    """cci_bbs_pack: W fp32 [O, C] -> (vals [O, C/G, K], idx uint8 [O, C/G, K])."""
    _dev(W)
    if W.dtype != torch.float32 or W.dim() != 2:
        raise TypeError("W must be a float32 [O, C] tensor")
    O, C = W.shape
    if G < 1 or C % G:
        raise ValueError("C must be a multiple of G")
    shape = (O, C // G, K)
    if out is None:
        vals = torch.empty(shape, dtype=val_dtype, device=W.device)
        idx = torch.empty(shape, dtype=torch.uint8, device=W.device)
    else:
        vals, idx = _out(out[0], shape, val_dtype, W.device), _out(out[1], shape, torch.uint8, W.device)
    _check(_lib.cci_bbs_pack(_ptr(W), O, C, G, K, _ptr(vals), _code(val_dtype), _ptr(idx), _stream(W)))
    return vals, idx


def _empty_2of4(M, R, device):
    if M % 16 or R % 64:
        raise ValueError("a 2:4 operand needs M % 16 == 0 and R % 64 == 0")
    return (torch.empty((R // 64, M // 16, 64, 8), dtype=torch.bfloat16, device=device),
            torch.empty((R // 64, M // 16, 64), dtype=torch.int16, device=device))


def bbs_to_2of4(vals: torch.Tensor, idx: torch.Tensor, G: int):
    """cci_bbs_to_2of4: balanced packing [O, C/G, K] -> prepared 2:4 operand
    (a_vals bf16 [C/64, O/16, 64, 8], a_idx int16 [C/64, O/16, 64] holding
    the uint16 index words) of the O x C matrix."""
    _dev(vals), _dev(idx)
    O, ng, K = vals.shape
    C = ng * G
    av, ai = _empty_2of4(O, C, vals.device)
    _check(_lib.cci_bbs_to_2of4(_ptr(vals), _code(vals.dtype), _ptr(idx), O, C, G, K, _ptr(av), _ptr(ai),
                                _stream(vals)))
    return av, ai


def to_2of4_transposed(vals: torch.Tensor, idx: torch.Tensor, G: int):
    """cci_to_2of4_transposed: CCI packing [O/G, K, C] of W_hat [O, C] ->
    prepared 2:4 operand of W_hat^T (rows C, reduction O)."""
    _dev(vals), _dev(idx)
    ng, K, C = vals.shape
    O = ng * G
    av, ai = _empty_2of4(C, O, vals.device)
    _check(_lib.cci_to_2of4_transposed(_ptr(vals), _code(vals.dtype), _ptr(idx), O, C, G, K, _ptr(av), _ptr(ai),
                                       _stream(vals)))
    return av, ai


def spmm_2of4(X: torch.Tensor, a_vals: torch.Tensor, a_idx: torch.Tensor, *, scale=None, bias=None, residual=None,
              relu=False, out_dtype=None, out=None) -> torch.Tensor:
    """cci_spmm_2of4: Y [N, M] = epilogue(X [N, R] . A^T) with A a prepared
    2:4 operand [M, R] (sparse matrix cores)."""
    _dev(X), _dev(a_vals), _dev(a_idx)
    N, R = X.shape
    ks, mbs, _, _ = a_vals.shape
    M = mbs * 16
    if ks * 64 != R or tuple(a_idx.shape) != (ks, mbs, 64) or a_vals.dtype != torch.bfloat16:
        raise ValueError("2:4 operand does not match X")
    if a_vals.device != X.device or a_idx.device != X.device:
        raise ValueError("X and the operand must be on one device")
    Y = _out(out, (N, M), out_dtype or X.dtype, X.device)
    ep = _epilogue(scale, bias, residual, relu, M, Y.shape, Y.dtype, X.device)
    _check(_lib.cci_spmm_2of4(_ptr(X), _code(X.dtype), N, R, _ptr(a_vals), _ptr(a_idx), M, ctypes.byref(ep), _ptr(Y),
                              _code(Y.dtype), _stream(X)))
    return Y


# ------------------------------------------------ improved targeted dropout --

def td_schedule(step: int, total: int, G: int, K: int):
    """cci_td_schedule: (candidates per group, candidate dropout rate)."""
    n = _i32()
    p = ctypes.c_double()
    _check(_lib.cci_td_schedule(step, total, G, K, ctypes.byref(n), ctypes.byref(p)))
    return n.value, p.value


def td_mask(W: torch.Tensor, G: int, n_target: int, bits: torch.Tensor, drop_rate: float, w_dtype=torch.bfloat16,
            out=None):
    """cci_td_mask: W fp32 [O, C], bits int32 [O, C] (the uint32 random words)
    -> (W_eff [O, C] of w_dtype, keep uint8 [O, C])."""
    _dev(W), _dev(bits)
    O, C = W.shape
    if W.dtype != torch.float32 or bits.dtype not in (torch.int32, torch.uint32) or tuple(bits.shape) != (O, C):
        raise ValueError("W must be float32 [O, C] and bits 32-bit [O, C]")
    if out is None:
        We = torch.empty((O, C), dtype=w_dtype, device=W.device)
        keep = torch.empty((O, C), dtype=torch.uint8, device=W.device)
    else:
        We, keep = _out(out[0], (O, C), w_dtype, W.device), _out(out[1], (O, C), torch.uint8, W.device)
    _check(_lib.cci_td_mask(_ptr(W), O, C, G, n_target, _ptr(bits), float(drop_rate), _ptr(We), _code(w_dtype),
                            _ptr(keep), _stream(W)))
    return We, keep


def grad_packed(dY: torch.Tensor, X: torch.Tensor, idx: torch.Tensor, G: int, out=None) -> torch.Tensor:
    """cci_grad_packed: dvals fp32 [O/G, K, C] from dY [N, O], X [N, C]."""
    _dev(dY), _dev(X), _dev(idx)
    N, O = dY.shape
    ng, K, C = idx.shape
    if X.shape != (N, C) or ng * G != O or X.dtype != dY.dtype or idx.dtype != torch.uint8:
        raise ValueError("shape or dtype mismatch")
    dv = _out(out, (ng, K, C), torch.float32, dY.device)
    _check(_lib.cci_grad_packed(_ptr(dY), _ptr(X), _code(dY.dtype), N, C, _ptr(idx), O, G, K, _ptr(dv), _stream(dY)))
    return dv


# ------------------------------------------------------ log2(G)-bit indices --

def index_width(G: int) -> int:
    """cci_index_width: ceil(log2 G), at least 1."""
    b = int(_lib.cci_index_width(G))
    if b < 0:
        raise ValueError("G outside [1, 256]")
    return b


def index_bits(idx: torch.Tensor, bits: int, out=None) -> torch.Tensor:
    """cci_index_bits: uint8 index array (any shape) -> int32 tensor holding
    the uint32 words of its `bits`-bit stream."""
    _dev(idx)
    if idx.dtype != torch.uint8:
        raise TypeError("idx must be uint8")
    n = idx.numel()
    nb = _sz()
    _check(_lib.cci_index_stream_bytes(n, bits, ctypes.byref(nb)))
    words = _out(out, (nb.value // 4,), torch.int32, idx.device)
    _check(_lib.cci_index_bits(_ptr(idx), n, bits, _ptr(words), _stream(idx)))
    return words


def spmm_bits(X: torch.Tensor, vals: torch.Tensor, idx: torch.Tensor, G: int, idx_bits: int, *, scale=None,
              bias=None, residual=None, relu=False, out_dtype=None, out=None) -> torch.Tensor:
    """cci_spmm_bits: the few-row (N <= 64) CCI product reading `idx_bits`-bit
    indices (the stream of index_bits, or the uint8 array for 8)."""
    _dev(X), _dev(vals), _dev(idx)
    N, C = X.shape
    ng, K, C2 = vals.shape
    if C2 != C:
        raise ValueError("shape mismatch between X and packed weights")
    O = ng * G
    Y = _out(out, (N, O), out_dtype or X.dtype, X.device)
    ep = _epilogue(scale, bias, residual, relu, O, Y.shape, Y.dtype, X.device)
    _check(_lib.cci_spmm_bits(_ptr(X), _code(X.dtype), N, C, _ptr(vals), _code(vals.dtype), _ptr(idx), idx_bits, O, G,
                              K, ctypes.byref(ep), _ptr(Y), _code(Y.dtype), _stream(X)))
    return Y
