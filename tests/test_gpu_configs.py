"""Parity of every workload configuration at its full size (the 4096-channel
layers c2 and c3-up are in test_gpu_large.py).

* c1 (512 x 512, 4-bit, 5 sweeps): the whole chain (Gram, grid, sweeps,
  exact objective) against the oracle on every entry, teacher-forced.
* c3-down (4096 x 11008, 3-bit, 10 sweeps): the whole 11008 x 11008 Gram
  over all 262144 tokens against the oracle's fp64 Gram of the same X; CD on
  all rows on that Sigma (the layer's own, damped, in fp32) against a seeded
  64-row sample, teacher-forced and free-running; and the same on the more
  strongly coupled Gram of a 2048-token prefix.
* c4 (4096 x 4096, 3-bit, s = 1% outliers, 10 iterations; c2's activations):
  the whole CD + IHT run on the layer's own Sigma (the oracle's Gram of all
  262144 tokens) against the oracle's whole run.  g must agree within 1e-4
  after every CD and IHT step.  P_s itself is an exact decision on the same
  fp32 V, so at full size it is checked on a seeded V (identical support).
  End to end, V is fp32 on the GPU and fp64 in the oracle; supports may then
  differ only at entries whose |V| lies within 1e-5 of the threshold.  The
  structured variant runs on a 2048-token prefix Gram.
* c5 (14848 x 59392, 4-bit, 5 sweeps): the Gram over 262144 device-drawn
  tokens streamed in 8192-token chunks, on every diagonal entry and a seeded
  256 x 256 block, against the oracle's fp64 sums of the same numbers; CD
  on all rows against a seeded 64-row sample, teacher-forced and
  free-running, on a Sigma with the workload's coupling; and a stress case on
  a rank-deficient Sigma (see the two tests).

Every CD input is a Sigma the oracle forms itself (no GPU output feeds the
oracle).  At c5 the fp64 Gram of all tokens would take the host about half
an hour, so its Sigma comes from a 256-token prefix (see the test); a prefix
Gram with fewer tokens than channels is more strongly coupled than a
workload's own (whose off-diagonal entries are about n^-1/2 of the
diagonal), which makes it the harder parity input."""
import numpy as np
import pytest
import torch

import synth
from parity import dev, free_running, host, rel_fro, teacher_forced

pytestmark = pytest.mark.gpu


def host_sigma(oracle, spec, tokens):
    X = synth.activations(spec, n=tokens)
    return oracle.damp(oracle.gram_blas(X), spec.damp)


def cd_row_sampled(qe, oracle, W, S32, bits, sweeps, rows, label, block=128, free=True,
                   code_frac=1e-3):
    """All rows on the GPU, the sampled rows in the oracle, both on the same
    fp32 Sigma and the same grid; teacher-forced (and free-running) checks."""
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
    T = W[rows].astype(np.float64) @ S64
    print(f"[{label}] teacher-forced oracle over {len(rows)} rows", flush=True)
    teacher_forced(oracle, W[rows], S64, bits, scale[rows], zero[rows], hist, whats, Rs, T=T,
                   label=label, code_frac=code_frac)
    if free:
        print(f"[{label}] free-running oracle", flush=True)
        free_running(oracle, W[rows], S64, bits, scale[rows], zero[rows], hist, whats, Rs, T=T,
                     label=label)


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
    hist, whats, Rs, objs = [], [], [], []
    flags = qe.QE_INIT_FROM_W
    for _ in range(spec.sweeps):
        obj = torch.zeros(1, dtype=torch.float64, device="cuda")
        qe.cd_sweep(Wd, dev(S32), spec.bits, scale_d, zero_d, Wh, codes, R, 1, flags=flags,
                    obj=obj)
        flags = qe.QE_R_VALID | qe.QE_CODES_VALID
        hist.append(host(codes).astype(np.int32))
        whats.append(host(Wh))
        Rs.append(host(R))
        objs.append(float(host(obj)[0]))
    S64 = S32.astype(np.float64)
    tf = teacher_forced(oracle, W, S64, spec.bits, scale, zero, hist, whats, Rs, gpu_obj=objs,
                        label="c1")
    free_running(oracle, W, S64, spec.bits, scale, zero, hist, whats, Rs, label="c1")
    exact = host(qe.objective(Wd, Wh, dev(S32)))
    f_last = oracle.objective(W, whats[-1], S64)
    assert exact[0] == pytest.approx(f_last, rel=1e-4)
    assert tf[-1]["obj_rel_err"] <= 1e-4
    assert exact[1] == pytest.approx(float(np.sum((W.astype(np.float64) @ S32) * W)), rel=1e-5)


@pytest.fixture(scope="module")
def c3down_x():
    spec = synth.CONFIGS["c3down"]
    print(f"[c3-down] drawing X {spec.p}x{spec.n}", flush=True)
    return synth.activations(spec)


@pytest.fixture(scope="module")
def c3down_sigma64(c3down_x, oracle):
    """The oracle's undamped fp64 Gram of all 262144 tokens (Lemma 1)."""
    p, n = c3down_x.shape
    S = np.zeros((p, p), np.float64)
    step = 32768
    for t0 in range(0, n, step):
        print(f"[c3-down] oracle Gram, tokens {t0}..{min(n, t0 + step)} of {n}", flush=True)
        oracle.gram_blas(c3down_x[:, t0:t0 + step], out=S)
    return S


@pytest.mark.timeout(900)
def test_c3_down_projection_gram_full_size(qe, c3down_x, c3down_sigma64):
    """The whole 11008 x 11008 Sigma against the oracle's fp64 Gram of all
    262144 tokens (relative Frobenius <= 1e-5), the diagonal entry by entry
    (outlier channels included), exactly symmetric."""
    Xd = dev(c3down_x)
    S = host(qe.gram(Xd))
    del Xd
    torch.cuda.empty_cache()
    assert np.array_equal(S, S.T)
    err = rel_fro(S, c3down_sigma64)
    print(f"[c3-down] Gram relative Frobenius error {err:.3e}", flush=True)
    assert err <= 1e-5
    d, dref = np.diag(S).astype(np.float64), np.diag(c3down_sigma64)
    assert np.max(np.abs(d - dref) / dref) <= 1e-5


@pytest.mark.timeout(900)
def test_c3_down_projection_own_sigma(qe, oracle, c3down_sigma64):
    spec = synth.CONFIGS["c3down"]
    W = synth.weights(spec)
    S32 = oracle.damp(c3down_sigma64, spec.damp).astype(np.float32)
    cd_row_sampled(qe, oracle, W, S32, spec.bits, spec.sweeps,
                   synth.row_sample(spec.q, 64, spec.cfg), "c3-down own Sigma")


@pytest.mark.timeout(900)
def test_c3_down_projection_prefix_sigma(qe, oracle):
    """The same layer on the Gram of a 2048-token prefix (damped 0.01):
    fewer tokens than channels, so its off-diagonal entries are about 11
    times the workload's relative to the diagonal."""
    spec = synth.CONFIGS["c3down"]
    W = synth.weights(spec)
    S32 = host_sigma(oracle, spec, 2048).astype(np.float32)
    cd_row_sampled(qe, oracle, W, S32, spec.bits, spec.sweeps,
                   synth.row_sample(spec.q, 64, spec.cfg), "c3-down 2048-token Sigma")


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


@pytest.mark.timeout(900)
def test_c4_outlier_full_run(qe, oracle, c2_sigma64):
    spec = synth.CONFIGS["c4"]
    c2 = synth.CONFIGS["c2"]
    x_seed = lambda sp: sp.cfg if sp.x_cfg is None else sp.x_cfg       # noqa: E731
    assert x_seed(spec) == x_seed(c2) and spec.p == c2.p and spec.n == c2.n   # c2's activations
    q, p, bits, iters, s = spec.q, spec.p, spec.bits, spec.sweeps, spec.s_budget
    W = synth.weights(spec)
    S32 = oracle.damp(c2_sigma64, spec.damp).astype(np.float32)     # the layer's own Sigma
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


@pytest.mark.timeout(900)
def test_c5_gram_full_size_streamed_sampled(qe, oracle):
    spec = synth.CONFIGS["c5"]
    p, n, chunk = spec.p, spec.n, 8192
    idx = synth.entry_sample(p, 256, spec.cfg)
    assert len(idx) >= 256
    ref_block = np.zeros((len(idx), len(idx)), np.float64)
    ref_diag = np.zeros(p, np.float64)
    every = np.arange(p)
    S = torch.empty((p, p), dtype=torch.float32, device="cuda")
    for c in range(n // chunk):
        if c % 8 == 0:
            print(f"[c5] Gram chunk {c} of {n // chunk}", flush=True)
        Xc = synth.activation_chunk_device(spec, c, chunk, "cuda")
        qe.gram(Xc, Sigma=S, accumulate=c > 0)
        Xh = host(Xc)                 # the very numbers the GPU used
        del Xc
        # the oracle's sums over this chunk's tokens, added up over chunks
        oracle.gram_blas(Xh[idx], out=ref_block)
        ref_diag += oracle.gram_entries(Xh, every, every)
        del Xh
    idx_d = torch.as_tensor(idx, device="cuda")
    block = host(S[idx_d][:, idx_d])
    blockT = host(S[:, idx_d][idx_d])
    diag = host(torch.diagonal(S))
    del S
    torch.cuda.empty_cache()
    assert np.array_equal(block, blockT.T)
    assert rel_fro(block, ref_block) <= 1e-5
    assert rel_fro(diag, ref_diag) <= 1e-5
    assert np.max(np.abs(diag - ref_diag) / ref_diag) <= 1e-5


C5_PREFIX = 256          # tokens of the c5 CD parity Sigma


def c5_prefix_gram(oracle, spec):
    X = synth.activation_chunk(spec, 0, tokens=C5_PREFIX)
    print(f"[c5] oracle Gram of a {C5_PREFIX}-token prefix", flush=True)
    return oracle.gram_blas(X, row_block=4096)


@pytest.mark.timeout(1200)
def test_c5_cd_row_sampled(qe, oracle):
    """c5 CD with the workload's coupling.  The fp64 Gram of all 262144
    tokens at p = 59392 would take the host about half an hour, so Sigma comes
    from a 256-token prefix; alone, that Gram has rank 256 and off-diagonal
    entries 1/16 of the diagonal (the workload's: 1/512 = n^-1/2, full rank,
    condition number about 8).  Damping by sqrt(262144 / 256) - 1 = 31 times
    the mean diagonal restores the workload's ratio of off-diagonal to
    diagonal entries and a condition number of about 10; the full bar
    applies."""
    spec = synth.CONFIGS["c5"]
    W = synth.weights(spec)
    S64 = c5_prefix_gram(oracle, spec)
    S32 = oracle.damp(S64, np.sqrt(spec.n / C5_PREFIX) - 1.0).astype(np.float32)
    del S64
    cd_row_sampled(qe, oracle, W, S32, spec.bits, spec.sweeps,
                   synth.row_sample(spec.q, 64, spec.cfg), "c5")


@pytest.mark.timeout(1200)
def test_c5_cd_stress_rank_deficient_sigma(qe, oracle):
    """Stress case: the 256-token prefix Gram with the workload's 0.01
    damping -- rank 256 of 59392, condition number about 26000, 32 times the
    workload's coupling.  A tie decision then moves a long stretch of the
    rest of its row (measured: about 10000 of 59392 codes), so the 0.1% cap,
    which presumes rare ties with short consequences, does not describe this
    input.  What is unique is checked instead: every code in which the GPU
    differs from the teacher-forced oracle is a tie decision or follows from
    earlier tie decisions of its row (parity.explain_row), and the objective
    agrees within 1e-4 after every sweep."""
    spec = synth.CONFIGS["c5"]
    W = synth.weights(spec)
    S32 = oracle.damp(c5_prefix_gram(oracle, spec), spec.damp).astype(np.float32)
    cd_row_sampled(qe, oracle, W, S32, spec.bits, spec.sweeps,
                   synth.row_sample(spec.q, 64, spec.cfg), "c5 stress", free=False,
                   code_frac=1.0)


@pytest.mark.timeout(900)
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
