"""GPU parity of the outlier-aware path (Sec. 4): P_s, lambda_max and the
full CD + IHT iteration, against the fp64 oracle.

P_s on the same fp32 V is an integer decision taken in the same precision by
both sides, so the support must be identical, ties and zeros included.
End to end, E is fp32 on the GPU and fp64 in the oracle; the supports must
still be identical on these seeds, and g must agree within 1e-4."""
import numpy as np
import pytest
import torch

import synth
from parity import dev, host

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("shape,s", [((512, 512), 2621), ((77, 301), 100), ((10, 10), 0),
                                     ((10, 10), 100), ((33, 7), 5), ((4096, 64), 20000)])
def test_topk_identical_support(qe, oracle, shape, s):
    V = synth.gaussian(shape, seed=1)
    V.reshape(-1)[::13] = 0.25          # exact ties in |v|
    V.reshape(-1)[7::29] = -0.25
    V.reshape(-1)[3::11] = 0.0          # exact zeros
    out, sup, nnz = qe.topk_abs(dev(V), s)
    n = int(host(nnz)[0])
    ref_sup, ref_dense = oracle.topk_abs(V, s)
    assert n == len(ref_sup)
    assert np.array_equal(host(sup)[:n], ref_sup)
    assert np.array_equal(host(out), ref_dense)


def test_lambda_max(qe, oracle):
    """An upper bound of the largest eigenvalue (Lemma 3 needs the step
    1/(2 lambda) with lambda >= lambda_max), tight to 1e-3."""
    X = synth.correlated_activations(300, 2000, 0.9, 3, out_channels=6, out_mult=20.0)
    S = oracle.damp(oracle.gram(X), 0.01).astype(np.float32)
    lam = qe.lambda_max(dev(S))
    ref = oracle.lambda_max(S)
    assert ref <= lam <= ref * (1 + 1e-3)


def _power_method(S, max_iters, tol):
    """The stop rule of qe_lambda_max in fp64: Rayleigh quotients of the unit
    iterates from 1/sqrt(p); the first one within tol (relative) of its
    predecessor, else the last; returned with its residual norm."""
    S = np.asarray(S, np.float64)
    v = np.full(S.shape[0], 1.0 / np.sqrt(S.shape[0]))
    prev = None
    for _ in range(max_iters):
        y = S @ v
        lam = float(v @ y)
        res = float(np.linalg.norm(y - lam * v))
        if prev is not None and abs(lam - prev) <= tol * lam:
            return lam, res
        prev = lam
        v = y / np.linalg.norm(y)
    return lam, res


@pytest.mark.parametrize("max_iters,tol", [(1, 1e-7), (3, 1e-7), (40, 1e-7), (500, 1e-2),
                                           (500, 1e-4)])
def test_lambda_max_stop_rule(qe, max_iters, tol):
    """Iteration counts and tolerances that stop inside, at the end of and
    across the 32-iteration host checks give the bound (quotient plus
    residual norm) of the same iteration as an fp64 power method with the
    same rule; once the iterates have converged, never less than the largest
    eigenvalue (early iterates bound some eigenvalue, not necessarily it)."""
    X = synth.correlated_activations(300, 2000, 0.9, 4, out_channels=6, out_mult=20.0)
    S = (X.astype(np.float64) @ X.T.astype(np.float64)).astype(np.float32)
    lam = qe.lambda_max(dev(S), max_iters=max_iters, tol=tol)
    rho, res = _power_method(S, max_iters, tol)
    assert lam == pytest.approx(rho + res, rel=2e-6)
    if max_iters >= 40:
        # converged iterates: the eigenvalue within the radius is the largest
        assert lam >= np.linalg.eigvalsh(S.astype(np.float64))[-1]


def run_outlier_gpu(qe, W, S32, bits, scale, zero, s, lam, sweeps, H0, sup0, n0, block=0,
                    extra=0):
    q, p = W.shape
    Wd, Sd = dev(W), dev(S32)
    Wh = torch.empty_like(Wd)
    codes = torch.zeros((q, p), dtype=torch.uint8, device="cuda")
    H = H0.clone()
    E = torch.empty_like(Wd)
    sup = sup0.clone()
    nnz = n0.clone()
    obj = torch.zeros(2 * sweeps, dtype=torch.float64, device="cuda")
    qe.cd_outlier_sweep(Wd, Sd, bits, dev(scale), dev(zero), Wh, codes, H, E, s, lam, sup, nnz,
                        sweeps, block=block, flags=qe.QE_INIT_FROM_W | extra, obj=obj)
    n = int(host(nnz)[0])
    return dict(What=host(Wh), codes=host(codes).astype(np.int32), H=host(H), E=host(E),
                support=host(sup)[:n], obj=host(obj))


@pytest.mark.parametrize("q,p,bits,frac,corr,fp32", [(512, 512, 3, 0.01, 0.9, False),
                                                      (512, 512, 3, 0.01, 0.9, True),
                                                      (96, 200, 3, 0.02, 0.5, False),
                                                      (130, 257, 2, 0.005, 0.9, False)])
def test_outlier_matches_oracle(qe, oracle, q, p, bits, frac, corr, fp32):
    W = synth.gaussian((q, p), seed=5, std=0.02)
    W.reshape(-1)[::487] *= 10.0
    X = synth.correlated_activations(p, 2048, corr, 6, out_channels=max(1, p // 100),
                                     out_mult=30.0)
    S = oracle.damp(oracle.gram(X), 0.01)
    S32 = S.astype(np.float32)
    s = int(frac * q * p)
    lam = float(np.float32(oracle.lambda_max(S32)))
    # initial outliers H = P_s(W) and the outlier-aware grid, both on the GPU
    H0, sup0, n0 = qe.topk_abs(dev(W), s)
    scale_d, zero_d = qe.grid_minmax(dev(W), bits, H0)
    ref_sup0, ref_H0 = oracle.topk_abs(W, s)
    assert np.array_equal(host(sup0)[:int(host(n0)[0])], ref_sup0)
    scale, zero = oracle.grid_minmax(W, bits, ref_H0)
    assert np.array_equal(host(scale_d), scale) and np.array_equal(host(zero_d), zero)

    sweeps = 4
    g = run_outlier_gpu(qe, W, S32, bits, scale, zero, s, lam, sweeps, H0, sup0, n0,
                        extra=qe.QE_CD_FP32 if fp32 else 0)
    ref = oracle.outlier(W, S32, bits, scale, zero, s, lam, sweeps)
    for k in range(sweeps):
        assert g["obj"][2 * k] == pytest.approx(ref.g_cd[k], rel=1e-4), f"g after CD, it {k + 1}"
        assert g["obj"][2 * k + 1] == pytest.approx(ref.g[k], rel=1e-4), f"g after IHT, it {k + 1}"
        assert g["obj"][2 * k + 1] <= g["obj"][2 * k] * (1 + 1e-6)       # Lemma 3
    assert np.array_equal(g["support"], ref.support)
    assert np.mean(g["codes"] != ref.codes) <= 1e-3
    assert np.allclose(g["H"], ref.H, rtol=1e-3, atol=1e-7)


def test_zero_budget_equals_plain_cd(qe, oracle):
    q, p = 64, 130
    W = synth.gaussian((q, p), seed=7, std=0.02)
    X = synth.correlated_activations(p, 1024, 0.9, 8)
    S32 = oracle.damp(oracle.gram(X), 0.01).astype(np.float32)
    scale, zero = oracle.grid_minmax(W, 3)
    Hz = torch.zeros((q, p), dtype=torch.float32, device="cuda")
    sup = torch.zeros(1, dtype=torch.int64, device="cuda")
    n0 = torch.zeros(1, dtype=torch.int64, device="cuda")
    g = run_outlier_gpu(qe, W, S32, 3, scale, zero, 0, 1.0, 3, Hz, sup, n0)
    Wd = dev(W)
    Wh = torch.empty_like(Wd)
    codes = torch.zeros((q, p), dtype=torch.uint8, device="cuda")
    R = torch.empty_like(Wd)
    qe.cd_sweep(Wd, dev(S32), 3, dev(scale), dev(zero), Wh, codes, R, 3)
    assert np.array_equal(g["What"], host(Wh))
    assert np.array_equal(g["codes"], host(codes).astype(np.int32))
    assert not np.any(g["H"])


# ---- structured (column) outliers, Sec. 4.3 "Structured Outliers"
@pytest.mark.parametrize("q,p,c", [(64, 300, 7), (512, 512, 5), (33, 70, 0), (40, 50, 60)])
def test_topk_columns_identical(qe, oracle, q, p, c):
    V = synth.gaussian((q, p), seed=41)
    V[:, 9] = V[:, 3]              # equal norms: the lower column is kept
    V[:, 17] = -V[:, 3]
    V[:, 5] = 0.0                  # all-zero columns are never kept
    c = min(c, p)
    out, cols, sup, nnz = qe.topk_columns(dev(V), c)
    ref_cols, ref_sup, ref_out = oracle.topk_columns(V, c)
    n = int(host(nnz)[0])
    assert n == len(ref_sup)
    assert np.array_equal(host(cols)[:len(ref_cols)], ref_cols)
    assert np.array_equal(host(sup)[:n], ref_sup)
    assert np.array_equal(host(out), ref_out)


@pytest.mark.parametrize("q,p,ncols,corr", [(256, 384, 6, 0.9), (96, 200, 3, 0.5)])
def test_structured_outlier_matches_oracle(qe, oracle, q, p, ncols, corr):
    W = synth.gaussian((q, p), seed=43, std=0.02)
    W[:, ::37] *= 8.0              # a few heavy columns
    X = synth.correlated_activations(p, 2048, corr, 44, out_channels=max(1, p // 100),
                                     out_mult=30.0)
    S32 = oracle.damp(oracle.gram(X), 0.01).astype(np.float32)
    s = ncols * q
    lam = float(np.float32(oracle.lambda_max(S32)))
    H0, cols0, sup0, n0 = qe.topk_columns(dev(W), ncols)
    ref_cols0, ref_sup0, ref_H0 = oracle.topk_columns(W, ncols)
    assert np.array_equal(host(cols0), ref_cols0)
    scale, zero = oracle.grid_minmax(W, 3, ref_H0)
    sweeps = 4
    Wd, Sd = dev(W), dev(S32)
    Wh = torch.empty_like(Wd)
    codes = torch.zeros((q, p), dtype=torch.uint8, device="cuda")
    E = torch.empty_like(Wd)
    sup = torch.zeros(s, dtype=torch.int64, device="cuda")
    sup[:int(host(n0)[0])] = sup0[:int(host(n0)[0])]
    obj = torch.zeros(2 * sweeps, dtype=torch.float64, device="cuda")
    qe.cd_outlier_sweep(Wd, Sd, 3, dev(scale), dev(zero), Wh, codes, H0, E, s, lam, sup, n0,
                        sweeps, flags=qe.QE_INIT_FROM_W | qe.QE_OUTLIER_COLUMNS, obj=obj)
    g = host(obj)
    ref = oracle.outlier(W, S32, 3, scale, zero, s, lam, sweeps, structured=True)
    for k in range(sweeps):
        assert g[2 * k] == pytest.approx(ref.g_cd[k], rel=1e-4), f"g after CD, it {k + 1}"
        assert g[2 * k + 1] == pytest.approx(ref.g[k], rel=1e-4), f"g after IHT, it {k + 1}"
        assert g[2 * k + 1] <= g[2 * k] * (1 + 1e-6)                  # Lemma 3
    n = int(host(n0)[0])
    assert np.array_equal(host(sup)[:n], ref.support)
    Hg = host(H0)
    assert np.array_equal(np.nonzero(np.any(Hg != 0, axis=0))[0],
                          np.nonzero(np.any(ref.H != 0, axis=0))[0])
    assert np.allclose(Hg, ref.H, rtol=1e-3, atol=1e-7)
    assert np.mean(host(codes).astype(np.int32) != ref.codes) <= 1e-3


def test_outlier_debug_checks_scan_h(qe, oracle):
    """QE_DEBUG_CHECKS in the outlier-aware call also scans H."""
    q, p, bits = 48, 96, 3
    W = synth.gaussian((q, p), seed=41, std=0.02)
    X = synth.correlated_activations(p, 512, 0.9, 42)
    S32 = oracle.damp(oracle.gram(X), 0.01).astype(np.float32)
    s = 40
    H, sup, nnz = qe.topk_abs(dev(W), s)
    Hh = host(H)
    Hh[host(sup)[0] // p, host(sup)[0] % p] = np.inf
    scale, zero = oracle.grid_minmax(W, bits, Hh)
    Wd, Sd = dev(W), dev(S32)
    Wh = torch.empty_like(Wd)
    E = torch.empty_like(Wd)
    codes = torch.zeros((q, p), dtype=torch.uint8, device="cuda")
    lam = float(np.float32(oracle.lambda_max(S32)))
    with pytest.raises(qe.QEError) as e:
        qe.cd_outlier_sweep(Wd, Sd, bits, dev(scale), dev(zero), Wh, codes, dev(Hh), E, s, lam,
                            sup, nnz, 2, flags=qe.QE_INIT_FROM_W | qe.QE_DEBUG_CHECKS)
    assert e.value.code == qe.QE_ERR_NONFINITE


def test_lemma3_descent_with_the_library_lambda(qe, oracle):
    """The whole outlier-aware run with the step size from qe_lambda_max:
    every IHT step keeps g from increasing (Lemma 3)."""
    q, p, bits, s, iters = 96, 256, 3, 300, 5
    W = synth.gaussian((q, p), seed=51, std=0.02)
    W.reshape(-1)[::41] *= 8.0
    X = synth.correlated_activations(p, 2048, 0.9, 52, out_channels=5, out_mult=20.0)
    S32 = oracle.damp(oracle.gram(X), 0.01).astype(np.float32)
    lam = qe.lambda_max(dev(S32))
    assert lam >= oracle.lambda_max(S32)
    H0, sup0, n0 = qe.topk_abs(dev(W), s)
    scale, zero = oracle.grid_minmax(W, bits, host(H0))
    g = run_outlier_gpu(qe, W, S32, bits, scale, zero, s, lam, iters, H0, sup0, n0)["obj"]
    for k in range(iters):
        assert g[2 * k + 1] <= g[2 * k] * (1 + 1e-6), f"IHT step {k + 1}"
        if k:
            assert g[2 * k] <= g[2 * k - 1] * (1 + 1e-6), f"CD step {k + 1}"
