"""Full-size parity on the 4096-channel layers, on the workload's own inputs,
in the launch configuration the benchmark times (block width 128).

The activations are the attention-projection workload's: 4096 x 262144
heavy-tailed tokens (128 x 2048, Student-t nu = 4, 1% outlier channels x30).
The MLP up-projection (11008 x 4096) draws the very same X, so both layers
share Sigma.

* Gram: the whole 4096 x 4096 Sigma against the oracle's fp64 Gram of all
  262144 tokens (relative Frobenius <= 1e-5), exactly symmetric -- from the
  channel-major X in one call, and from the token-major X streamed in chunks.
* CD on all rows of each layer, Sigma = the oracle's damped Gram of all
  262144 tokens cast to fp32 (Lemma 1: Sigma = X X^T over the calibration
  set); the oracle replays seeded row samples (512 rows of the attention
  projection, 128 of the up-projection; rows are independent, Sec. 3.2, so
  the sample is exact) teacher-forced after every sweep and free-running
  (tests/parity.py)."""
import numpy as np
import pytest
import torch

import synth
from parity import dev, free_running, host, rel_fro, teacher_forced

pytestmark = pytest.mark.gpu

SPEC = synth.CONFIGS["c2"]


@pytest.mark.timeout(900)
def test_gram_full_size_full_matrix(qe, c2_x, c2_sigma64):
    Xd = dev(c2_x)
    qe.gram(Xd)                              # code objects loaded
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    ev[0].record()
    Sd = qe.gram(Xd, check=False)
    ev[1].record()
    torch.cuda.synchronize()
    print(f"[c2] channel-major Gram: {ev[0].elapsed_time(ev[1]):.2f} ms", flush=True)
    S = host(Sd)
    del Xd, Sd
    torch.cuda.empty_cache()
    assert np.array_equal(S, S.T)
    err = rel_fro(S, c2_sigma64)
    print(f"[c2] Gram relative Frobenius error {err:.3e}", flush=True)
    assert err <= 1e-5
    # the diagonal (the CD step's divisors) entry by entry
    d, dref = np.diag(S).astype(np.float64), np.diag(c2_sigma64)
    assert np.max(np.abs(d - dref) / dref) <= 1e-5


@pytest.mark.timeout(900)
def test_gram_token_major_streamed_full_size(qe, c2_x, c2_sigma64):
    """Sec. 3.2 "Memory Footprint" (Sigma does not grow with n) and the
    calibration set of Sec. 5: the same 262144 tokens handed over token-major
    (n x p, the layout a model's activations come in) in chunks accumulated
    into Sigma, the first chunk ragged (30000 tokens, not a multiple of 32).
    The whole 4096 x 4096 Sigma against the oracle's fp64 Gram."""
    p, n = c2_x.shape
    cuts = [0, 30000] + list(range(30000 + 32768, n, 32768)) + [n]
    Sigma = torch.empty((p, p), dtype=torch.float32, device="cuda")
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    t = 0.0
    for c, (a, b) in enumerate(zip(cuts[:-1], cuts[1:])):
        chunk = dev(np.ascontiguousarray(c2_x[:, a:b].T))
        ev[0].record()
        qe.gram(chunk, layout=qe.QE_LAYOUT_NP, Sigma=Sigma, accumulate=c > 0)
        ev[1].record()
        torch.cuda.synchronize()
        t += ev[0].elapsed_time(ev[1]) * 1e-3
        del chunk
    S = host(Sigma)
    print(f"[c2] token-major Gram in {len(cuts) - 1} chunks: {t * 1e3:.2f} ms", flush=True)
    assert np.array_equal(S, S.T)
    assert rel_fro(S, c2_sigma64) <= 1e-5
    d, dref = np.diag(S).astype(np.float64), np.diag(c2_sigma64)
    assert np.max(np.abs(d - dref) / dref) <= 1e-5


def cd_rows_on_gpu(qe, W, S32, bits, sweeps, rows, block=128, extra=0):
    """All rows on the GPU, one sweep per call from What = W (extra: further
    flags, e.g. QE_CD_DENSE); the sampled rows' codes, What and R after every
    sweep."""
    q, p = W.shape
    scale, zero = qe.grid_minmax(dev(W), bits)
    Wd, Sd = dev(W), dev(S32)
    Wh = torch.empty_like(Wd)
    codes = torch.zeros((q, p), dtype=torch.uint8, device="cuda")
    R = torch.empty_like(Wd)
    flags = qe.QE_INIT_FROM_W | extra
    hist, whats, Rs = [], [], []
    rows_d = torch.as_tensor(rows, device="cuda")
    for _ in range(sweeps):
        qe.cd_sweep(Wd, Sd, bits, scale, zero, Wh, codes, R, 1, block=block, flags=flags)
        flags = qe.QE_R_VALID | qe.QE_CODES_VALID | extra
        hist.append(host(codes[rows_d]).astype(np.int32))
        whats.append(host(Wh[rows_d]))
        Rs.append(host(R[rows_d]))
    sc, ze = host(scale), host(zero)
    del Wd, Sd, Wh, codes, R
    torch.cuda.empty_cache()
    return sc, ze, hist, whats, Rs


def row_sampled_parity(qe, oracle, spec, W, S64, rows, label, extra=0):
    S32 = oracle.damp(S64, spec.damp).astype(np.float32)
    sc, ze, hist, whats, Rs = cd_rows_on_gpu(qe, W, S32, spec.bits, spec.sweeps, rows,
                                             extra=extra)
    # the grid is an exact fp32 decision on both sides
    scale, zero = oracle.grid_minmax(W, spec.bits)
    assert np.array_equal(sc, scale) and np.array_equal(ze, zero)
    Sc = S32.astype(np.float64)
    T = W[rows].astype(np.float64) @ Sc
    print(f"[{label}] teacher-forced oracle over {len(rows)} rows x {spec.sweeps} sweeps",
          flush=True)
    tf = teacher_forced(oracle, W[rows], Sc, spec.bits, scale[rows], zero[rows], hist, whats, Rs,
                        T=T, label=label)
    print(f"[{label}] free-running oracle", flush=True)
    fr = free_running(oracle, W[rows], Sc, spec.bits, scale[rows], zero[rows], hist, whats, Rs,
                      T=T, label=label)
    print(f"[{label}] teacher-forced code differences per sweep "
          f"{[r['code_diff_frac'] for r in tf]}; free-running {fr['code_diff_frac']} "
          f"({fr['split_rows']} split rows)", flush=True)


@pytest.mark.timeout(900)
def test_cd_full_size_own_sigma(qe, oracle, c2_sigma64):
    W = synth.weights(SPEC)
    rows = synth.row_sample(SPEC.q, 512, SPEC.cfg)
    row_sampled_parity(qe, oracle, SPEC, W, c2_sigma64, rows, "c2 own Sigma")


@pytest.mark.timeout(900)
def test_c3_up_projection_own_sigma(qe, oracle, c2_sigma64):
    spec = synth.CONFIGS["c3up"]
    assert spec.x_cfg == SPEC.cfg and spec.p == SPEC.p       # the same activations
    W = synth.weights(spec)
    rows = synth.row_sample(spec.q, 128, spec.cfg)
    row_sampled_parity(qe, oracle, spec, W, c2_sigma64, rows, "c3-up own Sigma")


@pytest.mark.timeout(900)
def test_cd_full_size_dense_block_updates(qe, oracle, c2_sigma64):
    """The configuration the benchmark's roofline times: every block update
    on the matrix cores (QE_CD_DENSE), on c2's own Sigma, 512 seeded rows
    against the oracle, teacher-forced and free-running."""
    W = synth.weights(SPEC)
    rows = synth.row_sample(SPEC.q, 512, SPEC.cfg)
    row_sampled_parity(qe, oracle, SPEC, W, c2_sigma64, rows, "c2 own Sigma, dense",
                       extra=qe.QE_CD_DENSE)


@pytest.mark.timeout(900)
def test_cd_full_size_benchmark_call(qe, oracle, c2_sigma64):
    """The benchmark's call (all 10 sweeps in one qe_cd_sweep from What = W,
    the objective after each) against 10 single-sweep calls that carry the
    objective in obj[0] (QE_OBJ_IN): What, codes, R and every objective
    bitwise the same; every reported objective within 1e-6 of the fp64
    objective of the GPU's own What over the whole layer (problem (1) with
    the damped Sigma, <What - W, (What - W) Sigma>)."""
    W = synth.weights(SPEC)
    S32 = oracle.damp(c2_sigma64, SPEC.damp).astype(np.float32)
    S64 = S32.astype(np.float64)
    q, p, bits, sweeps = SPEC.q, SPEC.p, SPEC.bits, SPEC.sweeps
    Wd, Sd = dev(W), dev(S32)
    scale, zero = qe.grid_minmax(Wd, bits)
    Wh, R = torch.empty_like(Wd), torch.empty_like(Wd)
    codes = torch.zeros((q, p), dtype=torch.uint8, device="cuda")
    obj = torch.zeros(sweeps, dtype=torch.float64, device="cuda")
    qe.cd_sweep(Wd, Sd, bits, scale, zero, Wh, codes, R, sweeps, block=128,
                flags=qe.QE_INIT_FROM_W, obj=obj)
    multi = (host(Wh), host(codes), host(R), host(obj))
    whats = []
    for k in range(sweeps):
        if k > 0:
            obj[k].copy_(obj[k - 1])
        qe.cd_sweep(Wd, Sd, bits, scale, zero, Wh, codes, R, 1, block=128,
                    flags=(qe.QE_INIT_FROM_W if k == 0
                           else qe.QE_R_VALID | qe.QE_CODES_VALID | qe.QE_OBJ_IN),
                    obj=obj[k:])
        whats.append(host(Wh))
    single = (whats[-1], host(codes), host(R), host(obj))
    del Wd, Sd, Wh, R, codes
    torch.cuda.empty_cache()
    for a, b, name in zip(multi, single, ("What", "codes", "R", "objective")):
        assert np.array_equal(a, b), name
    W64 = W.astype(np.float64)
    for k in range(sweeps):
        D = whats[k].astype(np.float64) - W64
        f = float(np.sum(D * (D @ S64)))
        err = abs(multi[3][k] - f) / f
        print(f"[c2 call] sweep {k + 1}: objective {multi[3][k]:.9e}, fp64 of What "
              f"{f:.9e}, rel. error {err:.2e}", flush=True)
        assert err <= 1e-6
