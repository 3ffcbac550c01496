"""ctypes binding of libqe.so (include/qe.h) on torch device tensors.

Argument marshalling only: every step of the QuantEase hot path runs in the
HIP kernels behind the C ABI; torch provides device memory and the stream.
There is no fallback: if libqe.so is missing or no GPU is present, the calls
raise.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Tuple

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libqe.so")

QE_OK = 0
QE_ERR_ARG = 1
QE_ERR_DIAG = 2
QE_ERR_SCALE = 3
QE_ERR_WORKSPACE = 4
QE_ERR_HIP = 5
QE_ERR_UNSUPPORTED = 6
QE_ERR_TOO_LARGE = 7
QE_ERR_NONFINITE = 8
QE_NOALLOC_SCRATCH_BYTES = 64 << 20

QE_LAYOUT_PN = 0
QE_LAYOUT_NP = 1
QE_GRAM_FP32 = 0x100
QE_GRAM_BF16X3 = 0x200

QE_INIT_FROM_W = 0x1
QE_R_VALID = 0x2
QE_CODES_VALID = 0x4
QE_RELAX_MASK = 0xff00
QE_OUTLIER_COLUMNS = 0x10
QE_CD_FP32 = 0x20
QE_CD_DENSE = 0x10000
QE_DEBUG_CHECKS = 0x40
QE_OBJ_IN = 0x80


def QE_RELAX_PERIOD(k: int) -> int:
    """Flag bits for relaxed sweeps every k-th sweep of a call (qe.h)."""
    return (int(k) & 0xff) << 8

_vp = ctypes.c_void_p
_i64 = ctypes.c_int64
_int = ctypes.c_int
_f32 = ctypes.c_float
_sz = ctypes.c_size_t

# name -> (restype, argtypes); mirrors include/qe.h
SIGNATURES = {
    "qe_status_string": (ctypes.c_char_p, [_int]),
    "qe_version": (_int, []),
    "qe_sync_status": (_int, [_vp, _vp]),
    "qe_gram_workspace_size": (_sz, [_i64, _i64]),
    "qe_gram": (_int, [_vp, _i64, _i64, _int, _vp, _int, _f32, _vp, _sz, _vp]),
    "qe_grid_minmax": (_int, [_vp, _vp, _i64, _i64, _int, _vp, _vp, _vp]),
    "qe_cd_workspace_size": (_sz, [_i64, _i64, _int]),
    "qe_cd_sweep": (_int, [_vp, _vp, _i64, _i64, _int, _vp, _vp, _vp, _vp, _vp, _int, _int,
                           ctypes.c_uint32, _vp, _vp, _sz, _vp]),
    "qe_cd_sweep_noalloc": (_int, [_vp, _vp, _i64, _i64, _int, _vp, _vp, _vp, _vp, _vp, _int,
                                   _int, ctypes.c_uint32, _vp, _vp, _vp]),
    "qe_outlier_workspace_size": (_sz, [_i64, _i64, _int, _i64]),
    "qe_cd_outlier_sweep": (_int, [_vp, _vp, _i64, _i64, _int, _vp, _vp, _vp, _vp, _vp, _vp,
                                   _i64, _f32, _vp, _vp, _int, _int, ctypes.c_uint32, _vp, _vp,
                                   _sz, _vp]),
    "qe_topk_workspace_size": (_sz, [_i64, _i64]),
    "qe_topk_abs": (_int, [_vp, _i64, _i64, _vp, _vp, _vp, _vp, _sz, _vp]),
    "qe_topk_columns_workspace_size": (_sz, [_i64, _i64]),
    "qe_topk_columns": (_int, [_vp, _i64, _i64, _i64, _vp, _vp, _vp, _vp, _vp, _sz, _vp]),
    "qe_packed_row_bytes": (_i64, [_i64, _int]),
    "qe_pack_codes": (_int, [_vp, _i64, _i64, _int, _vp, _vp]),
    "qe_outliers_csr": (_int, [_vp, _i64, _i64, _vp, _vp, _i64, _vp, _vp, _vp, _vp]),
    "qe_objective_workspace_size": (_sz, [_i64, _i64]),
    "qe_objective": (_int, [_vp, _vp, _vp, _vp, _i64, _i64, _vp, _vp, _sz, _vp]),
    "qe_lambda_workspace_size": (_sz, [_i64]),
    "qe_lambda_max": (_int, [_vp, _i64, _int, _f32, ctypes.POINTER(_f32), _vp, _sz, _vp]),
}

_lib = None


class QEError(RuntimeError):
    def __init__(self, code: int, where: str):
        self.code = code
        super().__init__(f"{where}: {status_string(code)} (status {code})")


def load() -> ctypes.CDLL:
    """Loads libqe.so (built in-tree by paper_2309_01885_amd/build.py)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python paper_2309_01885_amd/build.py` (no CPU fallback exists)")
        lib = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _lib = lib
    return _lib


def status_string(code: int) -> str:
    return load().qe_status_string(code).decode()


def _stream(stream=None) -> _vp:
    s = torch.cuda.current_stream() if stream is None else stream
    return _vp(s.cuda_stream)


def _ptr(t: Optional[torch.Tensor], dtype, name: str, numel: Optional[int] = None) -> _vp:
    if t is None:
        return _vp(None)
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if numel is not None and t.numel() != numel:
        raise ValueError(f"{name} must have {numel} elements, got {t.numel()}")
    return _vp(t.data_ptr())


def _check(code: int, where: str):
    if code != QE_OK:
        raise QEError(code, where)


def workspace(nbytes: int, device) -> torch.Tensor:
    """A device workspace; zero-filled, so that its status word reads QE_OK
    before any call has used it."""
    return torch.zeros(max(int(nbytes), 256), dtype=torch.uint8, device=device)


def sync_status(ws: torch.Tensor, stream=None) -> int:
    """Waits for the stream; returns (and clears) the workspace's device status word."""
    return load().qe_sync_status(_vp(ws.data_ptr()), _stream(stream))


def _finish(ws, check, where, stream=None):
    if check:
        _check(sync_status(ws, stream), where)


# ---------------------------------------------------------------------------- Gram
def gram(X: torch.Tensor, layout: int = QE_LAYOUT_PN, Sigma: Optional[torch.Tensor] = None,
         accumulate: bool = False, damp: float = 0.0, ws: Optional[torch.Tensor] = None,
         check: bool = True, stream=None, fp32: bool = False,
         bf16x3: bool = False) -> torch.Tensor:
    """Sigma (+)= X X^T (qe_gram).  fp32=True selects the fp32 matrix-core
    products (QE_GRAM_FP32), bf16x3=True the three-way bf16 split on every
    tile (QE_GRAM_BF16X3), instead of the default split products."""
    lib = load()
    if X.dim() != 2:
        raise ValueError("X must be 2-D")
    p, n = (X.shape if layout == QE_LAYOUT_PN else X.shape[::-1])
    if fp32:
        layout |= QE_GRAM_FP32
    if bf16x3:
        layout |= QE_GRAM_BF16X3
    if Sigma is None:
        Sigma = torch.empty((p, p), dtype=torch.float32, device=X.device)
    need = lib.qe_gram_workspace_size(p, n)
    if ws is None:
        ws = workspace(need, X.device)
    _check(lib.qe_gram(_ptr(X, torch.float32, "X"), p, n, layout,
                       _ptr(Sigma, torch.float32, "Sigma", p * p), 1 if accumulate else 0,
                       float(damp), _vp(ws.data_ptr()), ws.numel(), _stream(stream)), "qe_gram")
    _finish(ws, check, "qe_gram", stream)
    return Sigma


# ---------------------------------------------------------------------------- grid
def grid_minmax(W: torch.Tensor, bits: int, H: Optional[torch.Tensor] = None,
                stream=None) -> Tuple[torch.Tensor, torch.Tensor]:
    lib = load()
    q, p = W.shape
    scale = torch.empty(q, dtype=torch.float32, device=W.device)
    zero = torch.empty(q, dtype=torch.float32, device=W.device)
    _check(lib.qe_grid_minmax(_ptr(W, torch.float32, "W"), _ptr(H, torch.float32, "H", q * p)
                              if H is not None else _vp(None), q, p, bits,
                              _ptr(scale, torch.float32, "scale"), _ptr(zero, torch.float32, "zero"),
                              _stream(stream)), "qe_grid_minmax")
    return scale, zero


# ---------------------------------------------------------------------------- CD
def cd_workspace_size(q: int, p: int, block: int = 0) -> int:
    return int(load().qe_cd_workspace_size(q, p, block))


def cd_sweep(W, Sigma, bits, scale, zero, W_hat, codes, R, sweeps, block: int = 0,
             flags: int = QE_INIT_FROM_W, obj: Optional[torch.Tensor] = None,
             ws: Optional[torch.Tensor] = None, check: bool = True, stream=None):
    """In place on W_hat (fp32), codes (uint8) and R (fp32), all q x p."""
    lib = load()
    q, p = W.shape
    if ws is None:
        ws = workspace(cd_workspace_size(q, p, block), W.device)
    if obj is not None and (obj.dtype != torch.float64 or obj.numel() < sweeps):
        raise ValueError("obj must be a float64 device tensor with >= sweeps entries")
    _check(lib.qe_cd_sweep(_ptr(W, torch.float32, "W"), _ptr(Sigma, torch.float32, "Sigma", p * p),
                           q, p, bits, _ptr(scale, torch.float32, "scale", q),
                           _ptr(zero, torch.float32, "zero", q),
                           _ptr(W_hat, torch.float32, "W_hat", q * p),
                           _ptr(codes, torch.uint8, "codes", q * p),
                           _ptr(R, torch.float32, "R", q * p), sweeps, block, flags,
                           _ptr(obj, torch.float64, "obj") if obj is not None else _vp(None),
                           _vp(ws.data_ptr()), ws.numel(), _stream(stream)), "qe_cd_sweep")
    _finish(ws, check, "qe_cd_sweep", stream)
    return W_hat, codes, R


def cd_sweep_noalloc(W, Sigma, bits, scale, zero, W_hat, codes, R, sweeps, block: int = 0,
                     flags: int = QE_INIT_FROM_W, obj: Optional[torch.Tensor] = None,
                     status: Optional[torch.Tensor] = None, stream=None):
    """qe_cd_sweep_noalloc: as cd_sweep, with the library's fixed scratch in
    place of a workspace (nothing is allocated).  status: None or an int32
    device tensor of one element receiving the call's data-error status in
    stream order.  Calls that overlap on one GPU race (one shared scratch)."""
    lib = load()
    q, p = W.shape
    if obj is not None and (obj.dtype != torch.float64 or obj.numel() < sweeps):
        raise ValueError("obj must be a float64 device tensor with >= sweeps entries")
    _check(lib.qe_cd_sweep_noalloc(
        _ptr(W, torch.float32, "W"), _ptr(Sigma, torch.float32, "Sigma", p * p), q, p, bits,
        _ptr(scale, torch.float32, "scale", q), _ptr(zero, torch.float32, "zero", q),
        _ptr(W_hat, torch.float32, "W_hat", q * p), _ptr(codes, torch.uint8, "codes", q * p),
        _ptr(R, torch.float32, "R", q * p), sweeps, block, flags,
        _ptr(obj, torch.float64, "obj") if obj is not None else _vp(None),
        _ptr(status, torch.int32, "status", 1) if status is not None else _vp(None),
        _stream(stream)), "qe_cd_sweep_noalloc")
    return W_hat, codes, R


# ---------------------------------------------------------------------------- outlier-aware CD
def outlier_workspace_size(q: int, p: int, block: int, s: int) -> int:
    return int(load().qe_outlier_workspace_size(q, p, block, s))


def cd_outlier_sweep(W, Sigma, bits, scale, zero, W_hat, codes, H, E, s, lambda_max, support,
                     support_nnz, sweeps, block: int = 0, flags: int = QE_INIT_FROM_W,
                     obj: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None,
                     check: bool = True, stream=None):
    """In place on W_hat, codes, H, E, support (int64[s]) and support_nnz (int64[1])."""
    lib = load()
    q, p = W.shape
    if ws is None:
        ws = workspace(outlier_workspace_size(q, p, block, s), W.device)
    if obj is not None and (obj.dtype != torch.float64 or obj.numel() < 2 * sweeps):
        raise ValueError("obj must be a float64 device tensor with >= 2*sweeps entries")
    _check(lib.qe_cd_outlier_sweep(
        _ptr(W, torch.float32, "W"), _ptr(Sigma, torch.float32, "Sigma", p * p), q, p, bits,
        _ptr(scale, torch.float32, "scale", q), _ptr(zero, torch.float32, "zero", q),
        _ptr(W_hat, torch.float32, "W_hat", q * p), _ptr(codes, torch.uint8, "codes", q * p),
        _ptr(H, torch.float32, "H", q * p), _ptr(E, torch.float32, "E", q * p), int(s),
        float(lambda_max), _ptr(support, torch.int64, "support") if s > 0 else _vp(None),
        _ptr(support_nnz, torch.int64, "support_nnz", 1), sweeps, block, flags,
        _ptr(obj, torch.float64, "obj") if obj is not None else _vp(None),
        _vp(ws.data_ptr()), ws.numel(), _stream(stream)), "qe_cd_outlier_sweep")
    _finish(ws, check, "qe_cd_outlier_sweep", stream)
    return W_hat, codes, H, E


# ---------------------------------------------------------------------------- P_s
def topk_abs(V: torch.Tensor, s: int, ws: Optional[torch.Tensor] = None, check: bool = True,
             stream=None):
    """P_s(V) over all entries of V: returns (dense P_s(V), support int64[s], nnz int64[1])."""
    lib = load()
    count = V.numel()
    out = torch.empty_like(V)
    support = torch.zeros(max(int(s), 1), dtype=torch.int64, device=V.device)
    nnz = torch.zeros(1, dtype=torch.int64, device=V.device)
    if ws is None:
        ws = workspace(lib.qe_topk_workspace_size(count, s), V.device)
    _check(lib.qe_topk_abs(_ptr(V, torch.float32, "V"), count, int(s),
                           _ptr(out, torch.float32, "out"), _vp(support.data_ptr()),
                           _ptr(nnz, torch.int64, "nnz"), _vp(ws.data_ptr()), ws.numel(),
                           _stream(stream)), "qe_topk_abs")
    _finish(ws, check, "qe_topk_abs", stream)
    return out, support, nnz


def topk_columns(V: torch.Tensor, c: int, ws: Optional[torch.Tensor] = None,
                 check: bool = True, stream=None):
    """Structured projection of the q x p matrix V (c whole columns of largest
    l2 norm): returns (dense result, kept columns int64[c], support int64[q*c],
    nnz int64[1])."""
    lib = load()
    q, p = V.shape
    out = torch.empty_like(V)
    cols = torch.full((max(int(c), 1),), -1, dtype=torch.int64, device=V.device)
    support = torch.zeros(max(int(q * c), 1), dtype=torch.int64, device=V.device)
    nnz = torch.zeros(1, dtype=torch.int64, device=V.device)
    if ws is None:
        ws = workspace(lib.qe_topk_columns_workspace_size(q, p), V.device)
    _check(lib.qe_topk_columns(_ptr(V, torch.float32, "V"), q, p, int(c),
                               _ptr(out, torch.float32, "out"), _vp(cols.data_ptr()),
                               _vp(support.data_ptr()), _ptr(nnz, torch.int64, "nnz"),
                               _vp(ws.data_ptr()), ws.numel(), _stream(stream)),
           "qe_topk_columns")
    _finish(ws, check, "qe_topk_columns", stream)
    return out, cols, support, nnz


# ---------------------------------------------------------------------------- export
def pack_codes(codes: torch.Tensor, bits: int, stream=None) -> torch.Tensor:
    """q x p uint8 codes -> q x qe_packed_row_bytes(p, bits) uint8 bit streams."""
    lib = load()
    q, p = codes.shape
    out = torch.empty((q, int(lib.qe_packed_row_bytes(p, bits))), dtype=torch.uint8,
                      device=codes.device)
    _check(lib.qe_pack_codes(_ptr(codes, torch.uint8, "codes"), q, p, int(bits),
                             _vp(out.data_ptr()), _stream(stream)), "qe_pack_codes")
    return out


def outliers_csr(H: torch.Tensor, support: torch.Tensor, nnz: torch.Tensor, stream=None):
    """CSR (rowptr int64[q+1], cols int32[cap], vals float32[cap]) of the
    support entries of H; the first nnz entries of cols / vals are valid."""
    lib = load()
    q, p = H.shape
    cap = support.numel()
    rowptr = torch.empty(q + 1, dtype=torch.int64, device=H.device)
    cols = torch.empty(max(cap, 1), dtype=torch.int32, device=H.device)
    vals = torch.empty(max(cap, 1), dtype=torch.float32, device=H.device)
    _check(lib.qe_outliers_csr(_ptr(H, torch.float32, "H"), q, p,
                               _ptr(support, torch.int64, "support"), _ptr(nnz, torch.int64, "nnz"),
                               cap, _vp(rowptr.data_ptr()), _vp(cols.data_ptr()),
                               _vp(vals.data_ptr()), _stream(stream)), "qe_outliers_csr")
    return rowptr, cols, vals


# ---------------------------------------------------------------------------- objective
def objective(W, W_hat, Sigma, H: Optional[torch.Tensor] = None,
              ws: Optional[torch.Tensor] = None, check: bool = True, stream=None) -> torch.Tensor:
    """Device float64[2]: (||(W_hat + H - W) X||^2, ||W X||^2) through Sigma."""
    lib = load()
    q, p = W.shape
    out = torch.zeros(2, dtype=torch.float64, device=W.device)
    if ws is None:
        ws = workspace(lib.qe_objective_workspace_size(q, p), W.device)
    _check(lib.qe_objective(_ptr(W, torch.float32, "W"), _ptr(W_hat, torch.float32, "W_hat", q * p),
                            _ptr(H, torch.float32, "H", q * p) if H is not None else _vp(None),
                            _ptr(Sigma, torch.float32, "Sigma", p * p), q, p,
                            _ptr(out, torch.float64, "out"), _vp(ws.data_ptr()), ws.numel(),
                            _stream(stream)), "qe_objective")
    _finish(ws, check, "qe_objective", stream)
    return out


# ---------------------------------------------------------------------------- lambda_max
def lambda_max(Sigma: torch.Tensor, max_iters: int = 500, tol: float = 1e-7,
               ws: Optional[torch.Tensor] = None, stream=None) -> float:
    lib = load()
    p = Sigma.shape[0]
    if ws is None:
        ws = workspace(lib.qe_lambda_workspace_size(p), Sigma.device)
    out = _f32(0.0)
    _check(lib.qe_lambda_max(_ptr(Sigma, torch.float32, "Sigma", p * p), p, int(max_iters),
                             float(tol), ctypes.byref(out), _vp(ws.data_ptr()), ws.numel(),
                             _stream(stream)), "qe_lambda_max")
    return float(out.value)
