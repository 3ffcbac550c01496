"""Parity of every workload configuration at its full size.

* c1 (512 x 512, 4-bit, 5 sweeps): the whole chain (Gram, grid, sweeps,
  exact objective) against the oracle on every entry.
* c3 (11008 x 4096 and 4096 x 11008, 3-bit, 10 sweeps): CD on all rows; the
  oracle replays a seeded row sample with the same Sigma (rows are
  independent, Sec. 3.2).  The down-projection Gram is also checked at its
  full 11008 x 262144 size on sampled entries.
* c4 (4096 x 4096, 3-bit, s = 1% outliers, 10 iterations): the whole CD + IHT
  run against the oracle's whole run.  g must agree within 1e-4 after every
  CD and IHT step.  P_s itself is an exact decision on the same fp32 V, so
  at full size it is checked on a seeded V (identical support).  End to end,
  V is fp32 on the GPU and fp64 in the oracle; supports may then differ only
  at entries whose |V| lies within 1e-5 of the threshold.
* c5 (14848 x 59392, 4-bit, 5 sweeps): the Gram over 262144 device-drawn
  tokens streamed in 8192-token chunks (sampled entries against the
  oracle's dot products of the same numbers), and CD on all rows against a
  row sample.

CD comparisons use a Sigma formed on the host from the oracle side (a short
token prefix, damped), so no GPU output feeds the oracle.  Row samples are
compared as described in parity.check_row_sampled_sweeps: rows whose CD
trajectory splits at an exact tie are checked for validity, the others for
the objective."""
import numpy as np
import pytest
import torch

import synth
from parity import check_row_sampled_sweeps, dev, host, rel_fro

pytestmark = pytest.mark.gpu


def host_sigma(oracle, spec, tokens):
    X = synth.activations(spec, n=tokens)
    return oracle.damp(oracle.gram(X), spec.damp)


def cd_row_sampled(qe, oracle, W, S32, bits, sweeps, rows, block=128):
    """All rows on the GPU, the sampled rows in the oracle, both on the same
    fp32 Sigma; per-sweep checks."""
    q, p = W.shape
    scale, zero = oracle.grid_minmax(W, bits)
    Wd, Sd = dev(W), dev(S32)
    Wh = torch.empty_like(Wd)
    codes = torch.zeros((q, p), dtype=torch.uint8, device="cuda")
    R = torch.empty_like(Wd)
    flags = qe.QE_INIT_FROM_W
    hist, whats, Rs = [], [], []
    rows_d = torch.as_tensor(rows, device="cuda")
    for _ in range(sweeps):
        qe.cd_sweep(Wd, Sd, bits, dev(scale), dev(zero), Wh, codes, R, 1, block=block,
                    flags=flags)
        flags = qe.QE_R_VALID | qe.QE_CODES_VALID
        hist.append(host(codes[rows_d]).astype(np.int32))
        whats.append(host(Wh[rows_d]))
        Rs.append(host(R[rows_d]))
    del Wd, Sd, Wh, codes, R
    torch.cuda.empty_cache()
    # the oracle takes the same fp32 Sigma, promoted
    S64 = S32.astype(np.float64)
    ref = oracle.cd(W[rows], S64, bits, scale[rows], zero[rows], sweeps)
    check_row_sampled_sweeps(W[rows], S64, whats, Rs, hist, ref)


def test_c1_whole_chain(qe, oracle):
    spec = synth.CONFIGS["c1"]
    W = synth.weights(spec)
    X = synth.activations(spec)
    S = host(qe.gram(dev(X), damp=spec.damp))
    S_ref = oracle.damp(oracle.gram(X), spec.damp)
    assert rel_fro(S, S_ref) <= 1e-5
    scale_d, zero_d = qe.grid_minmax(dev(W), spec.bits)
    scale, zero = oracle.grid_minmax(W, spec.bits)
    assert np.array_equal(host(scale_d), scale) and np.array_equal(host(zero_d), zero)
    # CD from the oracle's Sigma (fp32), all rows on both sides
    S32 = S_ref.astype(np.float32)
    Wd = dev(W)
    Wh = torch.empty_like(Wd)
    codes = torch.zeros(W.shape, dtype=torch.uint8, device="cuda")
    R = torch.empty_like(Wd)
    obj = torch.zeros(spec.sweeps, dtype=torch.float64, device="cuda")
    qe.cd_sweep(Wd, dev(S32), spec.bits, scale_d, zero_d, Wh, codes, R, spec.sweeps, obj=obj)
    ref = oracle.cd(W, S32.astype(np.float64), spec.bits, scale, zero, spec.sweeps)
    assert np.allclose(host(obj), ref.obj, rtol=1e-4)
    assert np.mean(host(codes).astype(np.int32) != ref.codes) <= 1e-3
    exact = host(qe.objective(Wd, Wh, dev(S32)))
    assert exact[0] == pytest.approx(ref.obj[-1], rel=1e-4)
    assert exact[1] == pytest.approx(float(np.sum((W.astype(np.float64) @ S32) * W)), rel=1e-5)


def test_c3_up_projection_row_sampled(qe, oracle):
    spec = synth.CONFIGS["c3up"]
    W = synth.weights(spec)
    S32 = host_sigma(oracle, spec, 2048).astype(np.float32)   # activations of the 4096-wide layer
    cd_row_sampled(qe, oracle, W, S32, spec.bits, spec.sweeps,
                   synth.row_sample(spec.q, 64, spec.cfg))


def test_c3_down_projection_gram_full_size_sampled(qe, oracle):
    spec = synth.CONFIGS["c3down"]
    X = synth.activations(spec)
    S = qe.gram(dev(X))
    idx = synth.entry_sample(spec.p, 128, spec.cfg, must=synth.outlier_channels(spec)[:16])
    ia, ib = np.meshgrid(idx, idx, indexing="ij")
    diag = synth.row_sample(spec.p, 1024, spec.cfg)
    ia = np.concatenate([ia.reshape(-1), diag])
    ib = np.concatenate([ib.reshape(-1), diag])
    got = host(S[torch.as_tensor(ia, device="cuda"), torch.as_tensor(ib, device="cuda")])
    del S
    torch.cuda.empty_cache()
    ref = oracle.gram_entries(X, ia, ib)
    assert rel_fro(got, ref) <= 1e-5


def test_c3_down_projection_row_sampled(qe, oracle):
    spec = synth.CONFIGS["c3down"]
    W = synth.weights(spec)
    S32 = host_sigma(oracle, spec, 2048).astype(np.float32)
    cd_row_sampled(qe, oracle, W, S32, spec.bits, spec.sweeps,
                   synth.row_sample(spec.q, 24, spec.cfg))


def test_c4_topk_full_size_identical(qe, oracle):
    spec = synth.CONFIGS["c4"]
    V = synth.gaussian((spec.q, spec.p), seed=11, std=0.05)
    V.reshape(-1)[::1009] = 0.125           # exact ties around the threshold region
    V.reshape(-1)[5::2003] = -0.125
    V.reshape(-1)[3::97] = 0.0
    s = spec.s_budget
    out, sup, nnz = qe.topk_abs(dev(V), s)
    n = int(host(nnz)[0])
    ref_sup, ref_dense = oracle.topk_abs(V, s)
    assert n == len(ref_sup) == s
    assert np.array_equal(host(sup)[:n], ref_sup)
    assert np.array_equal(host(out), ref_dense)


def test_c4_outlier_full_run(qe, oracle):
    spec = synth.CONFIGS["c4"]
    q, p, bits, iters, s = spec.q, spec.p, spec.bits, spec.sweeps, spec.s_budget
    W = synth.weights(spec)
    S32 = host_sigma(oracle, spec, 2048).astype(np.float32)
    lam = float(np.float32(oracle.lambda_max(S32)))
    H0, sup0, n0 = qe.topk_abs(dev(W), s)
    ref_sup0, ref_H0 = oracle.topk_abs(W, s)
    assert np.array_equal(host(sup0)[:int(host(n0)[0])], ref_sup0)
    scale, zero = oracle.grid_minmax(W, bits, ref_H0)
    Wd, Sd = dev(W), dev(S32)
    Wh = torch.empty_like(Wd)
    codes = torch.zeros((q, p), dtype=torch.uint8, device="cuda")
    E = torch.empty_like(Wd)
    obj = torch.zeros(2 * iters, dtype=torch.float64, device="cuda")
    qe.cd_outlier_sweep(Wd, Sd, bits, dev(scale), dev(zero), Wh, codes, H0, E, s, lam, sup0, n0,
                        iters, block=128, flags=qe.QE_INIT_FROM_W, obj=obj)
    g = host(obj)
    sup = host(sup0)[:int(host(n0)[0])]
    codes_g = host(codes).astype(np.int32)
    del Wd, Sd, Wh, codes, E
    torch.cuda.empty_cache()
    ref = oracle.outlier(W, S32, bits, scale, zero, s, lam, iters)
    for k in range(iters):
        assert g[2 * k] == pytest.approx(ref.g_cd[k], rel=1e-4), f"g after CD, it {k + 1}"
        assert g[2 * k + 1] == pytest.approx(ref.g[k], rel=1e-4), f"g after IHT, it {k + 1}"
        assert g[2 * k + 1] <= g[2 * k] * (1 + 1e-6)                  # Lemma 3
    assert np.mean(codes_g != ref.codes) <= 1e-3
    assert len(sup) == len(ref.support) == s
    diff = np.setxor1d(sup, ref.support)
    tau = ref.tau[-1]
    near = np.abs(np.abs(ref.V_last.reshape(-1)[diff]) - tau) <= 1e-5 * tau
    assert np.all(near), f"{len(diff)} support differences, {int(np.sum(~near))} away from tau"


def test_c5_gram_full_size_streamed_sampled(qe, oracle):
    spec = synth.CONFIGS["c5"]
    p, n, chunk = spec.p, spec.n, 8192
    idx = synth.entry_sample(p, 64, spec.cfg)
    diag = synth.row_sample(p, 512, spec.cfg)
    keep = np.unique(np.concatenate([idx, diag]))
    pos = {int(c): k for k, c in enumerate(keep)}
    keep_d = torch.as_tensor(keep, device="cuda")
    Xs = np.empty((len(keep), n), np.float32)
    S = torch.empty((p, p), dtype=torch.float32, device="cuda")
    for c in range(n // chunk):
        Xc = synth.activation_chunk_device(spec, c, chunk, "cuda")
        qe.gram(Xc, Sigma=S, accumulate=c > 0)
        Xs[:, c * chunk:(c + 1) * chunk] = host(Xc[keep_d])
        del Xc
    ia, ib = np.meshgrid(idx, idx, indexing="ij")
    ia = np.concatenate([ia.reshape(-1), diag])
    ib = np.concatenate([ib.reshape(-1), diag])
    got = host(S[torch.as_tensor(ia, device="cuda"), torch.as_tensor(ib, device="cuda")])
    sym = host(S[torch.as_tensor(ib, device="cuda"), torch.as_tensor(ia, device="cuda")])
    del S
    torch.cuda.empty_cache()
    assert np.array_equal(got, sym)
    la = np.array([pos[int(a)] for a in ia])
    lb = np.array([pos[int(b)] for b in ib])
    ref = oracle.gram_entries(Xs, la, lb)
    assert rel_fro(got, ref) <= 1e-5


def test_c5_cd_row_sampled(qe, oracle):
    spec = synth.CONFIGS["c5"]
    W = synth.weights(spec)
    X = synth.activation_chunk(spec, 0, tokens=256).astype(np.float64)
    # library product on the host side, in row blocks (one product of all
    # 59392^2 outputs overflows the BLAS library's 32-bit indexing)
    S64 = np.empty((spec.p, spec.p), np.float64)
    for r0 in range(0, spec.p, 4096):
        S64[r0:r0 + 4096] = X[r0:r0 + 4096] @ X.T
    del X
    S32 = oracle.damp(S64, spec.damp).astype(np.float32)
    del S64
    cd_row_sampled(qe, oracle, W, S32, spec.bits, spec.sweeps,
                   synth.row_sample(spec.q, 16, spec.cfg))


def test_c4_structured_outlier_run(qe, oracle):
    """The outlier-aware configuration with structured outliers (Sec. 4.3):
    floor(s / q) = 40 whole columns, 4 iterations against the oracle."""
    spec = synth.CONFIGS["c4"]
    q, p, bits, s = spec.q, spec.p, spec.bits, spec.s_budget
    iters = 4
    W = synth.weights(spec)
    S32 = host_sigma(oracle, spec, 2048).astype(np.float32)
    lam = float(np.float32(oracle.lambda_max(S32)))
    ncols = s // q
    H0, cols0, sup_c, n0 = qe.topk_columns(dev(W), ncols)
    ref_cols0, _, ref_H0 = oracle.topk_columns(W, ncols)
    assert np.array_equal(host(cols0), ref_cols0)
    scale, zero = oracle.grid_minmax(W, bits, ref_H0)
    Wd, Sd = dev(W), dev(S32)
    Wh = torch.empty_like(Wd)
    codes = torch.zeros((q, p), dtype=torch.uint8, device="cuda")
    E = torch.empty_like(Wd)
    sup = torch.zeros(s, dtype=torch.int64, device="cuda")
    n = int(host(n0)[0])
    sup[:n] = sup_c[:n]
    obj = torch.zeros(2 * iters, dtype=torch.float64, device="cuda")
    qe.cd_outlier_sweep(Wd, Sd, bits, dev(scale), dev(zero), Wh, codes, H0, E, s, lam, sup, n0,
                        iters, block=128, flags=qe.QE_INIT_FROM_W | qe.QE_OUTLIER_COLUMNS,
                        obj=obj)
    g = host(obj)
    Hcols = np.nonzero(np.any(host(H0) != 0, axis=0))[0]
    codes_g = host(codes).astype(np.int32)
    del Wd, Sd, Wh, codes, E
    torch.cuda.empty_cache()
    ref = oracle.outlier(W, S32, bits, scale, zero, s, lam, iters, structured=True)
    for k in range(iters):
        assert g[2 * k] == pytest.approx(ref.g_cd[k], rel=1e-4), f"g after CD, it {k + 1}"
        assert g[2 * k + 1] == pytest.approx(ref.g[k], rel=1e-4), f"g after IHT, it {k + 1}"
        assert g[2 * k + 1] <= g[2 * k] * (1 + 1e-6)                  # Lemma 3
    assert np.array_equal(Hcols, np.nonzero(np.any(ref.H != 0, axis=0))[0])
    assert np.mean(codes_g != ref.codes) <= 1e-3
