"""QuantEase CPU oracle (arXiv 2309.01885) -- TEST INFRASTRUCTURE ONLY.

A plain, slow, obviously-correct restatement of what the QuantEase hot path
computes, used to check the HIP library.  Only ``tests/``, the smoke check in
``__graft_entry__`` and the CPU-baseline leg of ``bench.py`` may import it; the
product package never does, and this module imports nothing from it.

Floating point is fp64 throughout (the paper does not fix a precision), except
``grid_minmax``: it decides an integer (the zero point) from floating-point
values, so it takes that decision in the kernel's precision, fp32.

Heavy loops live in ``qe_oracle.c`` (fp64, OpenMP over independent rows); this
module orchestrates them in the paper's order.  Library primitives used as
single steps: numpy matmul (the products W Sigma, (W - H) Sigma, D Sigma) and
``numpy.linalg.eigvalsh`` (the largest eigenvalue of Sigma).

Parity pins for every function are in ``tests/test_oracle_*.py``.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libqe_oracle.so")
_lib = None

_f32p = ctypes.POINTER(ctypes.c_float)
_f64p = ctypes.POINTER(ctypes.c_double)
_i32p = ctypes.POINTER(ctypes.c_int32)
_i64p = ctypes.POINTER(ctypes.c_int64)
_u8p = ctypes.POINTER(ctypes.c_uint8)
_i64 = ctypes.c_int64


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        from . import build as _build
        _build.build()
    _lib = bind(_LIB_PATH)
    return _lib


def bind(path: str) -> ctypes.CDLL:
    """Loads a build of qe_oracle.c from ``path`` and declares its signatures
    (the tests also bind deliberately broken copies of the source, to show
    that the pins catch each such mistake)."""
    lib = ctypes.CDLL(path)
    lib.qeo_gram.argtypes = [_f32p, _i64, _i64, ctypes.c_int, _f64p]
    lib.qeo_gram.restype = None
    lib.qeo_gram_entries.argtypes = [_f32p, _i64, _i64, ctypes.c_int, _i64p, _i64p, _i64, _f64p]
    lib.qeo_gram_entries.restype = None
    lib.qeo_grid_minmax.argtypes = [_f32p, _i64, _i64, ctypes.c_int, _f32p, _f32p, _f32p]
    lib.qeo_grid_minmax.restype = None
    lib.qeo_cd_sweep_lemma1.argtypes = [_f64p, _f64p, _i64, _i64, ctypes.c_int, _f64p, _f64p,
                                        _f64p, _i32p, _u8p, _f64p, ctypes.c_int, _i64]
    lib.qeo_cd_sweep_lemma1.restype = ctypes.c_int
    lib.qeo_cd_sweep_alg1.argtypes = [_f64p, _f64p, _i64, _i64, ctypes.c_int, _f64p, _f64p,
                                      _f64p, _i32p, _u8p, _f64p]
    lib.qeo_cd_sweep_alg1.restype = ctypes.c_int
    lib.qeo_cd_sweep_alg2.argtypes = [_f64p, _f64p, _i64, _i64, ctypes.c_int, _f64p, _f64p,
                                      _f64p, _i32p, _u8p, _f64p, _f64p]
    lib.qeo_cd_sweep_alg2.restype = None
    lib.qeo_topk_abs.argtypes = [_f64p, _i64, _i64, _i64p]
    lib.qeo_topk_abs.restype = _i64
    lib.qeo_num_threads.argtypes = []
    lib.qeo_num_threads.restype = ctypes.c_int
    return lib


def num_threads() -> int:
    """OpenMP threads the oracle's loops use."""
    return int(_load().qeo_num_threads())


def cd_sweep_timed(W, Sigma, bits, scale, zero, sweeps: int = 1) -> float:
    """Wall seconds of `sweeps` Lemma-1 sweeps from What = W, clocked around
    the C calls only (T = W Sigma is formed before the clock starts)."""
    import time
    lib = _load()
    W = np.asarray(W)
    q, p = W.shape
    S = _c(Sigma, np.float64)
    T = _c(np.asarray(W, np.float64) @ S, np.float64)
    Wh = _c(W, np.float64).copy()
    codes = np.zeros((q, p), np.int32)
    valid = np.zeros((q, p), np.uint8)
    sc = _c(scale, np.float32).astype(np.float64)
    ze = _c(zero, np.float32).astype(np.float64)
    dt = 0.0
    for _ in range(sweeps):
        t0 = time.perf_counter()
        rc = lib.qeo_cd_sweep_lemma1(_p(T, _f64p), _p(S, _f64p), q, p, bits, _p(sc, _f64p),
                                     _p(ze, _f64p), _p(Wh, _f64p), _p(codes, _i32p),
                                     _p(valid, _u8p), None, 0, 0)
        dt += time.perf_counter() - t0
        if rc != 0:
            raise ValueError("Sigma has a non-positive diagonal entry")
    return dt


def _p(a: np.ndarray, ptype):
    return a.ctypes.data_as(ptype)


def _c(a, dtype) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=dtype)


# --------------------------------------------------------------------------
# Gram matrix (Lemma 1: Sigma = X X^T) and damping
# --------------------------------------------------------------------------
def gram(X: np.ndarray, layout: int = 0) -> np.ndarray:
    """Sigma = X X^T in fp64.  ``layout`` 0: X is p x n; 1: X is n x p."""
    X = _c(X, np.float32)
    p, n = (X.shape if layout == 0 else X.shape[::-1])
    out = np.empty((p, p), dtype=np.float64)
    _load().qeo_gram(_p(X, _f32p), p, n, layout, _p(out, _f64p))
    return out


def gram_blas(X: np.ndarray, layout: int = 0, chunk: int = 8192, out=None,
              row_block: int = 8192) -> np.ndarray:
    """Sigma = X X^T in fp64 through the library product (numpy's BLAS), one
    token chunk at a time: Sigma = sum_c X_c X_c^T, each chunk promoted to
    fp64 (and, for very wide layers, row_block output rows per product).
    The same definition as ``gram``; for layers too large for the plain
    loops.  ``out`` (p x p fp64), if given, is accumulated into."""
    X = np.asarray(X)
    p, n = (X.shape if layout == 0 else X.shape[::-1])
    S = np.zeros((p, p), np.float64) if out is None else out
    for t0 in range(0, n, chunk):
        Xc = (X[:, t0:t0 + chunk] if layout == 0 else X[t0:t0 + chunk].T).astype(np.float64)
        for r0 in range(0, p, row_block):
            S[r0:r0 + row_block] += Xc[r0:r0 + row_block] @ Xc.T
    return S


def gram_entries(X: np.ndarray, ia, ib, layout: int = 0) -> np.ndarray:
    """Entries (ia[e], ib[e]) of X X^T, each a single fp64 dot product."""
    X = _c(X, np.float32)
    p, n = (X.shape if layout == 0 else X.shape[::-1])
    ia = _c(ia, np.int64)
    ib = _c(ib, np.int64)
    out = np.empty(ia.shape[0], dtype=np.float64)
    _load().qeo_gram_entries(_p(X, _f32p), p, n, layout, _p(ia, _i64p), _p(ib, _i64p),
                             ia.shape[0], _p(out, _f64p))
    return out


def damp(Sigma: np.ndarray, damp_frac: float) -> np.ndarray:
    """Sigma + damp_frac * mean(diag Sigma) * I.

    Not in the paper; the reading adopted for the workloads (a relative
    diagonal damping, so that Sigma_jj > 0 as Lemma 1 requires)."""
    S = np.array(Sigma, dtype=np.float64, copy=True)
    if damp_frac > 0.0:
        mean_diag = float(np.sum(np.diag(S))) / S.shape[0]
        S[np.diag_indices_from(S)] += damp_frac * mean_diag
    return S


# --------------------------------------------------------------------------
# Grid
# --------------------------------------------------------------------------
def grid_minmax(W: np.ndarray, bits: int, H: Optional[np.ndarray] = None):
    """Per-row asymmetric min/max grid (scale, zero) in fp32; entries with
    H != 0 are excluded (outlier-aware grid)."""
    W = _c(W, np.float32)
    q, p = W.shape
    scale = np.empty(q, dtype=np.float32)
    zero = np.empty(q, dtype=np.float32)
    Hp = None
    if H is not None:
        H = _c(H, np.float32)
        Hp = _p(H, _f32p)
    _load().qeo_grid_minmax(_p(W, _f32p), q, p, bits, Hp, _p(scale, _f32p), _p(zero, _f32p))
    return scale, zero


def dequant(codes: np.ndarray, scale: np.ndarray, zero: np.ndarray) -> np.ndarray:
    """Grid value s_i (k - z_i) of each code, fp64."""
    return np.asarray(scale, np.float64)[:, None] * (np.asarray(codes, np.float64)
                                                     - np.asarray(zero, np.float64)[:, None])


# --------------------------------------------------------------------------
# Export for serving: bit-packed codes and the outliers in CSR form.  The
# paper leaves serving kernels out of scope (Sec. 4.3, "Structured
# Outliers"); the layout here is this library's: each row of codes is one
# little-endian bit stream, code j in bits [j*bits, (j+1)*bits), bytes
# filled from their least significant bit; rows start on a byte boundary.
# --------------------------------------------------------------------------
def packed_row_bytes(p: int, bits: int) -> int:
    return (p * bits + 7) // 8


def pack_codes(codes: np.ndarray, bits: int) -> np.ndarray:
    """q x p codes in [0, 2^bits) -> q x packed_row_bytes(p, bits) uint8."""
    codes = np.asarray(codes, np.int64)
    q, p = codes.shape
    stream = ((codes[:, :, None] >> np.arange(bits)) & 1).reshape(q, p * bits).astype(np.uint8)
    pad = packed_row_bytes(p, bits) * 8 - p * bits
    stream = np.concatenate([stream, np.zeros((q, pad), np.uint8)], axis=1)
    return np.packbits(stream, axis=1, bitorder="little")


def unpack_codes(packed: np.ndarray, p: int, bits: int) -> np.ndarray:
    bitsarr = np.unpackbits(np.asarray(packed, np.uint8), axis=1, bitorder="little")
    stream = bitsarr[:, :p * bits].reshape(-1, p, bits).astype(np.int64)
    return np.sum(stream << np.arange(bits), axis=2)


def outliers_csr(H: np.ndarray, support: np.ndarray):
    """The support entries of H (q x p; support = ascending linear indices)
    as CSR: row pointers int64[q + 1], column indices int32, values float32."""
    H = np.asarray(H)
    q, p = H.shape
    support = np.asarray(support, np.int64)
    rows, cols = support // p, support % p
    rowptr = np.zeros(q + 1, np.int64)
    np.add.at(rowptr, rows + 1, 1)
    return np.cumsum(rowptr), cols.astype(np.int32), H[rows, cols].astype(np.float32)


# --------------------------------------------------------------------------
# Objective (problem (1) of Sec. 2.1) and relative calibration error (Sec. 3.4)
# --------------------------------------------------------------------------
def objective(W, What, Sigma, H=None) -> float:
    """f = ||W X - (What + H) X||_F^2 written through Sigma = X X^T:
    f = tr(D Sigma D^T) with D = What + H - W."""
    D = np.asarray(What, np.float64) - np.asarray(W, np.float64)
    if H is not None:
        D = D + np.asarray(H, np.float64)
    S = np.asarray(Sigma, np.float64)
    return float(np.sum((D @ S) * D))


def rel_error(W, What, Sigma, H=None) -> float:
    """||WX - What X||^2 / ||WX||^2, both written through Sigma."""
    Wd = np.asarray(W, np.float64)
    den = float(np.sum((Wd @ np.asarray(Sigma, np.float64)) * Wd))
    return objective(W, What, Sigma, H) / den


# --------------------------------------------------------------------------
# Coordinate descent (Sec. 3)
# --------------------------------------------------------------------------
@dataclass
class CDResult:
    What: np.ndarray                      # q x p fp64, final
    codes: np.ndarray                     # q x p int32, final
    valid: np.ndarray                     # q x p uint8
    obj: List[float] = field(default_factory=list)          # f after each sweep
    codes_hist: List[np.ndarray] = field(default_factory=list)
    margin_hist: List[np.ndarray] = field(default_factory=list)
    what_hist: List[np.ndarray] = field(default_factory=list)


def cd(W, Sigma, bits: int, scale, zero, sweeps: int, *, W0=None, codes0=None,
       codes_valid: bool = False, form: str = "lemma1", target=None,
       relax_period: int = 0, record: bool = True, obj_H=None, T=None, start_col: int = 0,
       with_obj: bool = True) -> CDResult:
    """Cyclic CD sweeps of QuantEase.

    W: q x p weights; Sigma: p x p (used as given, promoted to fp64);
    scale, zero: the per-row grid; W0: initial What (default W, Sec. 3.1);
    codes0/codes_valid: grid codes of W0 when W0 is on the grid.
    form: 'lemma1' (direct closed form), 'alg1' (rank-1 bookkeeping),
    'alg2' (accelerated partial update).  target: the matrix whose product
    with Sigma forms the linear term (W by default; W - H in the outlier-aware
    CD step).  relax_period k > 0: sweeps k, 2k, ... (1-based) write beta
    unquantized; the last sweep is always quantized.
    obj_H: H added to What in the recorded objective (outlier variant).
    T: the product target @ Sigma (fp64), if the caller already holds it
    (several calls on the same layer); formed here otherwise.
    start_col (lemma1 form, one sweep): begin the sweep at that column, the
    earlier coordinates counting as already visited.  with_obj=False skips
    the objective after each sweep.
    """
    if start_col and (form != "lemma1" or sweeps != 1):
        raise ValueError("start_col applies to one sweep of the lemma1 form")
    lib = _load()
    W = np.asarray(W)
    q, p = W.shape
    S = _c(Sigma, np.float64)
    tgt = np.asarray(W if target is None else target, np.float64)
    Wh = _c(W if W0 is None else W0, np.float64).copy()
    codes = np.zeros((q, p), np.int32) if codes0 is None else _c(codes0, np.int32).copy()
    valid = np.full((q, p), 1 if codes_valid else 0, np.uint8)
    sc = _c(scale, np.float32).astype(np.float64)
    ze = _c(zero, np.float32).astype(np.float64)
    res = CDResult(What=Wh, codes=codes, valid=valid)

    if form == "lemma1" or form == "alg1":
        T = _c(tgt @ S if T is None else T, np.float64)
    elif form == "alg2":
        d = np.diag(S).copy()
        N = S / d[None, :]                     # Sigma^norm_{:,j} = Sigma_{:,j} / Sigma_jj
        P = _c(tgt @ N, np.float64)            # P = W Sigma^norm, before zeroing the diagonal
        N = _c(N, np.float64)
        N[np.diag_indices_from(N)] = 0.0       # then Sigma^norm_jj = 0
        dW = np.empty((q, p), np.float64)
        Phat = np.empty((q, p), np.float64)
    else:
        raise ValueError(form)

    for k in range(1, sweeps + 1):
        relax = relax_period > 0 and k % relax_period == 0 and k != sweeps
        margin = np.empty((q, p), np.float64) if record else None
        if form == "lemma1":
            rc = lib.qeo_cd_sweep_lemma1(_p(T, _f64p), _p(S, _f64p), q, p, bits, _p(sc, _f64p),
                                         _p(ze, _f64p), _p(Wh, _f64p), _p(codes, _i32p),
                                         _p(valid, _u8p),
                                         _p(margin, _f64p) if margin is not None else None,
                                         1 if relax else 0, int(start_col))
            if rc != 0:
                raise ValueError("Sigma has a non-positive diagonal entry")
        elif form == "alg1":
            if relax:
                raise ValueError("relaxed sweeps are only provided in the lemma1 form")
            M = _c(Wh @ S, np.float64)
            rc = lib.qeo_cd_sweep_alg1(_p(T, _f64p), _p(S, _f64p), q, p, bits, _p(sc, _f64p),
                                       _p(ze, _f64p), _p(Wh, _f64p), _p(codes, _i32p),
                                       _p(valid, _u8p), _p(M, _f64p))
            if rc != 0:
                raise ValueError("Sigma has a non-positive diagonal entry")
        else:
            if relax:
                raise ValueError("relaxed sweeps are only provided in the lemma1 form")
            lib.qeo_cd_sweep_alg2(_p(P, _f64p), _p(N, _f64p), q, p, bits, _p(sc, _f64p),
                                  _p(ze, _f64p), _p(Wh, _f64p), _p(codes, _i32p),
                                  _p(valid, _u8p), _p(dW, _f64p), _p(Phat, _f64p))
        if with_obj:
            res.obj.append(objective(W, Wh, S, obj_H))
        if record:
            res.codes_hist.append(codes.copy())
            res.margin_hist.append(margin)
            res.what_hist.append(Wh.copy())
    return res


# --------------------------------------------------------------------------
# Outlier-aware QuantEase (Sec. 4, Algorithm "Outlier-Aware QuantEase")
# --------------------------------------------------------------------------
def topk_abs(V: np.ndarray, s: int):
    """P_s(V): the s entries largest in |V| (ties: lower linear index first;
    zeros never selected).  Returns (support as ascending linear indices,
    dense P_s(V) in V's dtype)."""
    V = np.asarray(V)
    flat = _c(V.reshape(-1), np.float64)
    sup = np.empty(max(int(s), 1), np.int64)
    nnz = _load().qeo_topk_abs(_p(flat, _f64p), flat.shape[0], int(s), _p(sup, _i64p))
    if nnz < 0:
        raise MemoryError("topk_abs")
    sup = sup[:nnz].copy()
    out = np.zeros(V.size, dtype=V.dtype)
    out[sup] = V.reshape(-1)[sup]
    return sup, out.reshape(V.shape)


def column_keys(V: np.ndarray) -> np.ndarray:
    """Squared l2 norm of every column of V, summed in fp64 and rounded to
    fp32: the selection key of the structured projection (both sides take
    that integer decision on the same fp32 key)."""
    V = np.asarray(V, np.float64)
    return np.sum(V * V, axis=0).astype(np.float32)


def topk_columns(V: np.ndarray, c: int):
    """Structured P (Sec. 4.3, "Structured Outliers"): keep the c columns of V
    with the largest l2 norm (ties: lower column index first; all-zero
    columns never kept), zero elsewhere.  Returns (kept columns ascending,
    support as ascending linear indices of every entry of those columns,
    dense result in V's dtype)."""
    V = np.asarray(V)
    q, p = V.shape
    cols, _ = topk_abs(column_keys(V), c)
    sup = (np.arange(q, dtype=np.int64)[:, None] * p + cols[None, :]).reshape(-1)
    out = np.zeros_like(V)
    out[:, cols] = V[:, cols]
    return cols, sup, out


def lambda_max(Sigma) -> float:
    """Largest eigenvalue of the symmetric matrix Sigma (fp64 eigvalsh)."""
    return float(np.linalg.eigvalsh(np.asarray(Sigma, np.float64))[-1])


@dataclass
class OutlierResult:
    What: np.ndarray
    H: np.ndarray
    codes: np.ndarray
    support: np.ndarray
    g_cd: List[float] = field(default_factory=list)     # g after the CD sweep of iteration k
    g: List[float] = field(default_factory=list)        # g after the IHT step of iteration k
    support_hist: List[np.ndarray] = field(default_factory=list)
    codes_hist: List[np.ndarray] = field(default_factory=list)
    margin_hist: List[np.ndarray] = field(default_factory=list)
    tau: List[float] = field(default_factory=list)      # s-th largest |V| of iteration k
    V_last: Optional[np.ndarray] = None                 # V of the last IHT step


def outlier_init(W, s: int, structured: bool = False):
    """H = P_s(W), What = W - H (Sec. 4.3, initialisation).  structured: the
    column projection with floor(s / q) columns instead of P_s."""
    Wd = np.asarray(W, np.float64)
    if structured:
        _, sup, H = topk_columns(Wd, int(s) // Wd.shape[0])
    else:
        sup, H = topk_abs(Wd, s)
    return sup, H, Wd - H


def outlier(W, Sigma, bits: int, scale, zero, s: int, lam: float, sweeps: int,
            record: bool = True, structured: bool = False) -> OutlierResult:
    """Block coordinate descent of Sec. 4.3: per iteration, one CD sweep on
    What with H fixed (target W - H), then one IHT step
    H <- P_s(H - eta grad_H g), grad_H g = 2 (H + What - W) Sigma, eta = 1/(2 lam).
    structured: P_s is replaced by the column projection keeping the
    floor(s / q) columns of largest l2 norm ("Structured Outliers", Sec. 4.3).
    ``scale``/``zero`` must be the outlier-aware grid (outliers of W excluded)."""
    W = np.asarray(W)
    Wd = W.astype(np.float64)
    S = _c(Sigma, np.float64)
    q = W.shape[0]
    sup, H, Wh = outlier_init(W, s, structured)
    q, p = W.shape
    codes = np.zeros((q, p), np.int32)
    res = OutlierResult(What=Wh, H=H, codes=codes, support=sup)
    eta = 1.0 / (2.0 * float(lam))
    for it in range(sweeps):
        # What starts off the grid (W - H); from the second iteration on every
        # code is valid, so the modified-CD tie rule applies.
        cres = cd(W, S, bits, scale, zero, 1, W0=Wh, codes0=codes, codes_valid=it > 0,
                  target=Wd - H, record=record, obj_H=H)
        Wh, codes = cres.What, cres.codes
        res.g_cd.append(cres.obj[0])
        grad = 2.0 * ((H + Wh - Wd) @ S)
        V = H - eta * grad
        if structured:
            _, sup, H = topk_columns(V, int(s) // q)
        else:
            sup, H = topk_abs(V, s)
        res.g.append(objective(Wd, Wh, S, H))
        res.tau.append(float(np.min(np.abs(V.reshape(-1)[sup]))) if len(sup) else 0.0)
        if it == sweeps - 1:
            res.V_last = V
        if record:
            res.support_hist.append(sup)
            res.codes_hist.append(codes.copy())
            res.margin_hist.append(cres.margin_hist[0])
    res.What, res.H, res.codes, res.support = Wh, H, codes, sup
    return res
