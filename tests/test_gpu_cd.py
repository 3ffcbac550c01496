"""GPU parity of qe_cd_sweep (Sec. 3: Lemma 1, the rank-1 identity, blocked)
against the fp64 oracle, on the same seeded fp32 inputs.

Bar (tests/parity.py), on every row of each case:
* teacher-forced, after every sweep: the oracle runs that sweep from the
  GPU's state after the previous one; at most 0.1% of codes differ, every
  row's first difference sits at an oracle tie (within 1e-4 grid units of a
  rounding boundary), and the objective -- the library's reported value and
  <What - W, R> from the GPU's residual -- agrees within 1e-4 relative;
* free-running: first divergences only at ties, identical rows agree on the
  objective, split rows keep descending.
Exact cases (weights on the grid, diagonal Sigma, constructed ties) must
match bit for bit.  The block-update products run on the split bf16 matrix
cores by default; the main parity cases also run with QE_CD_FP32 (fp32
matrix cores)."""
import json
import os

import numpy as np
import pytest
import torch

import synth
from parity import dev, free_running, host, teacher_forced

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def gpu_cd(qe, W, S32, bits, scale, zero, sweeps, block=0, per_sweep=True, W0=None, codes0=None,
           extra=0):
    q, p = W.shape
    Wd, Sd = dev(W), dev(S32)
    sc, ze = dev(scale), dev(zero)
    Wh = torch.empty_like(Wd)
    codes = torch.zeros((q, p), dtype=torch.uint8, device="cuda")
    R = torch.empty_like(Wd)
    flags = qe.QE_INIT_FROM_W
    if W0 is not None:
        Wh.copy_(dev(W0))
        flags = 0
        if codes0 is not None:
            codes.copy_(dev(codes0.astype(np.uint8)))
            flags = qe.QE_CODES_VALID
    flags |= extra
    hist, objs, whats, Rs = [], [], [], []
    if per_sweep:
        # one call per sweep, the objective carried from call to call (QE_OBJ_IN)
        obj = torch.zeros(1, dtype=torch.float64, device="cuda")
        for k in range(sweeps):
            qe.cd_sweep(Wd, Sd, bits, sc, ze, Wh, codes, R, 1, block=block, flags=flags, obj=obj)
            flags = qe.QE_R_VALID | qe.QE_CODES_VALID | qe.QE_OBJ_IN | extra
            hist.append(host(codes).astype(np.int32))
            objs.append(float(host(obj)[0]))
            whats.append(host(Wh))
            Rs.append(host(R))
    else:
        obj = torch.zeros(sweeps, dtype=torch.float64, device="cuda")
        qe.cd_sweep(Wd, Sd, bits, sc, ze, Wh, codes, R, sweeps, block=block, flags=flags, obj=obj)
        objs = list(host(obj))
        hist.append(host(codes).astype(np.int32))
    return dict(What=host(Wh), codes=host(codes).astype(np.int32), R=host(R), hist=hist,
                obj=objs, whats=whats, Rs=Rs)


def layer(q, p, n, seed, corr=0.0, bits=4, damp=0.01, spec="c1"):
    if corr > 0:
        X = synth.correlated_activations(p, n, corr, seed, out_channels=max(1, p // 50),
                                         out_mult=20.0)
        W = synth.gaussian((q, p), seed=seed, std=0.02)
    else:
        sp = synth.CONFIGS[spec]
        X = synth.activations(sp, n=n, p=p)
        W = synth.weights(sp, q=q, p=p)
    return W, X


def compare_sweeps(oracle, W, S32, bits, scale, zero, g, label, W0=None, codes0=None,
                   codes_valid0=False):
    """Teacher-forced and free-running comparison of a per-sweep GPU run over
    all rows of the layer."""
    S64 = S32.astype(np.float64)
    T = W.astype(np.float64) @ S64
    kw = dict(W0=W0, codes0=codes0, codes_valid0=codes_valid0, T=T, label=label)
    teacher_forced(oracle, W, S64, bits, scale, zero, g["hist"], g["whats"], g["Rs"],
                   gpu_obj=g["obj"], **kw)
    return free_running(oracle, W, S64, bits, scale, zero, g["hist"], g["whats"], g["Rs"], **kw)


def check_parity(oracle, W, S32, bits, scale, zero, g, label):
    return compare_sweeps(oracle, W, S32, bits, scale, zero, g, label)


@pytest.mark.parametrize("fp32", [False, True])
@pytest.mark.parametrize("q,p,corr,bits", [
    (512, 512, 0.0, 4),       # the small single-layer workload
    (512, 512, 0.9, 4),       # correlated channels: CD really moves
    (77, 200, 0.9, 3),        # ragged rows and a ragged last block
    (130, 301, 0.5, 2),
    (1, 33, 0.9, 4),
    (256, 768, 0.9, 4),       # aligned: the unguarded split-product loop
])
def test_cd_matches_oracle(qe, oracle, q, p, corr, bits, fp32):
    W, X = layer(q, p, 2048, 11, corr=corr, bits=bits)
    S32 = oracle.damp(oracle.gram(X), 0.01).astype(np.float32)
    scale, zero = oracle.grid_minmax(W, bits)
    sweeps = 5
    g = gpu_cd(qe, W, S32, bits, scale, zero, sweeps, extra=qe.QE_CD_FP32 if fp32 else 0)
    check_parity(oracle, W, S32, bits, scale, zero, g, f"cd {q}x{p} corr={corr} b={bits} fp32={fp32}")


@pytest.mark.parametrize("bits", [1, 8])
def test_extreme_bit_widths(qe, oracle, bits):
    """The narrowest and widest grids the ABI takes (2 and 256 levels)."""
    W, X = layer(128, 300, 1024, 41, corr=0.9, bits=bits)
    S32 = oracle.damp(oracle.gram(X), 0.01).astype(np.float32)
    scale, zero = oracle.grid_minmax(W, bits)
    g = gpu_cd(qe, W, S32, bits, scale, zero, 4)
    check_parity(oracle, W, S32, bits, scale, zero, g, f"bits {bits}")


def test_degenerate_rows(qe, oracle):
    """An all-zero row (grid [-1, 1], Sec. 2.1 reading), a constant row, a row
    with one nonzero entry and an ordinary row: the grid bit for bit, then
    the sweeps through the parity protocol."""
    W, X = layer(4, 96, 512, 42, corr=0.9)
    W[0] = 0.0
    W[1] = 0.5
    W[2] = 0.0
    W[2, 17] = -0.03
    S32 = oracle.damp(oracle.gram(X), 0.01).astype(np.float32)
    sc_d, ze_d = qe.grid_minmax(dev(W), 4)
    scale, zero = oracle.grid_minmax(W, 4)
    assert np.array_equal(host(sc_d), scale) and np.array_equal(host(ze_d), zero)
    g = gpu_cd(qe, W, S32, 4, scale, zero, 3)
    check_parity(oracle, W, S32, 4, scale, zero, g, "degenerate rows")
    assert np.all(g["What"][0] == 0.0)       # zero is a level of every grid


@pytest.mark.parametrize("q,p", [(1, 1), (1, 5), (5, 1), (3, 2)])
def test_tiny_layers(qe, oracle, q, p):
    """Single rows and columns: one panel, a partial block, no GEMM tile
    beyond the first."""
    W, X = layer(q, p, 64, 43 + q + p, corr=0.5)
    S32 = oracle.damp(oracle.gram(X), 0.01).astype(np.float32)
    scale, zero = oracle.grid_minmax(W, 3)
    g = gpu_cd(qe, W, S32, 3, scale, zero, 3)
    check_parity(oracle, W, S32, 3, scale, zero, g, f"tiny {q}x{p}")


@pytest.mark.parametrize("block", [16, 32, 64, 128])
def test_block_width_invariance(qe, oracle, block):
    W, X = layer(96, 250, 1024, 12, corr=0.9)
    S32 = oracle.damp(oracle.gram(X), 0.01).astype(np.float32)
    scale, zero = oracle.grid_minmax(W, 4)
    g = gpu_cd(qe, W, S32, 4, scale, zero, 4, block=block)
    check_parity(oracle, W, S32, 4, scale, zero, g, f"block {block}")


def test_multi_sweep_call_equals_resumed_calls(qe, oracle):
    W, X = layer(200, 260, 1024, 13, corr=0.9)
    S32 = oracle.damp(oracle.gram(X), 0.01).astype(np.float32)
    scale, zero = oracle.grid_minmax(W, 3)
    a = gpu_cd(qe, W, S32, 3, scale, zero, 4, per_sweep=True)
    b = gpu_cd(qe, W, S32, 3, scale, zero, 4, per_sweep=False)
    assert np.array_equal(a["What"], b["What"])
    assert np.array_equal(a["codes"], b["codes"])
    assert np.array_equal(a["R"], b["R"])
    assert a["obj"] == b["obj"]


def test_objective_paths_agree(qe, oracle):
    """The per-sweep objective is the incoming one plus the exact change of
    the sweep's coordinate moves (Lemma 1's one-dimensional quadratic).  The
    incoming value comes three ways: 0 from What = W (one multi-sweep call),
    carried in obj[0] (QE_OBJ_IN, per-sweep calls: bitwise the same as the
    multi-sweep call), or one pass <What - W, R> at the start of each resumed
    call.  All three follow the fp64 objective of the GPU's own What after
    every sweep, on a ragged shape (partial panel block and GEMM tiles)."""
    W, X = layer(150, 333, 1024, 31, corr=0.9)
    S32 = oracle.damp(oracle.gram(X), 0.01).astype(np.float32)
    scale, zero = oracle.grid_minmax(W, 4)
    sweeps = 5
    multi = gpu_cd(qe, W, S32, 4, scale, zero, sweeps, per_sweep=False)
    carried = gpu_cd(qe, W, S32, 4, scale, zero, sweeps, per_sweep=True)
    assert multi["obj"] == carried["obj"]
    Wd, Sd, sc, ze = dev(W), dev(S32), dev(scale), dev(zero)
    Wh, R = torch.empty_like(Wd), torch.empty_like(Wd)
    codes = torch.zeros(W.shape, dtype=torch.uint8, device="cuda")
    flags = qe.QE_INIT_FROM_W
    for k in range(sweeps):
        obj = torch.zeros(1, dtype=torch.float64, device="cuda")
        qe.cd_sweep(Wd, Sd, 4, sc, ze, Wh, codes, R, 1, flags=flags, obj=obj)
        flags = qe.QE_R_VALID | qe.QE_CODES_VALID
        f_ref = oracle.objective(W, carried["whats"][k], S32)
        assert np.array_equal(host(Wh), carried["whats"][k])
        f_pass = float(host(obj)[0])
        print(f"sweep {k + 1}: f {f_ref:.9e}, carried rel err "
              f"{abs(carried['obj'][k] - f_ref) / f_ref:.2e}, start-pass rel err "
              f"{abs(f_pass - f_ref) / f_ref:.2e}")
        assert carried["obj"][k] == pytest.approx(f_ref, rel=1e-5)
        assert f_pass == pytest.approx(f_ref, rel=1e-5)


def test_deterministic(qe, oracle):
    W, X = layer(256, 384, 1024, 14, corr=0.9)
    S32 = oracle.damp(oracle.gram(X), 0.01).astype(np.float32)
    scale, zero = oracle.grid_minmax(W, 4)
    a = gpu_cd(qe, W, S32, 4, scale, zero, 3, per_sweep=False)
    b = gpu_cd(qe, W, S32, 4, scale, zero, 3, per_sweep=False)
    assert np.array_equal(a["What"], b["What"]) and np.array_equal(a["R"], b["R"])


@pytest.mark.parametrize("fp32", [False, True])
@pytest.mark.parametrize("q,p", [(150, 270), (256, 512)])
def test_residual_is_exact_after_sweeps(qe, oracle, q, p, fp32):
    W, X = layer(q, p, 1024, 15, corr=0.9)
    S32 = oracle.damp(oracle.gram(X), 0.01).astype(np.float32)
    scale, zero = oracle.grid_minmax(W, 4)
    g = gpu_cd(qe, W, S32, 4, scale, zero, 3, extra=qe.QE_CD_FP32 if fp32 else 0)
    R_ref = (g["What"].astype(np.float64) - W) @ S32.astype(np.float64)
    scale_R = np.abs(g["What"].astype(np.float64) - W) @ np.abs(S32.astype(np.float64))
    assert np.all(np.abs(g["R"] - R_ref) <= 1e-5 * scale_R + 1e-30)


def block_update_regimes(hist, q, p, tile=128, super_w=256, rows_max=64, row_nz_max=32):
    """For every sweep that starts from valid codes, the number of (row tile,
    super-block) block updates that take the sparse path and the dense one,
    worked out from the codes alone: a tile's rows may each have changed at
    most row_nz_max codes of the super-block, and at most rows_max rows any."""
    out = []
    for k in range(1, len(hist)):
        moved = hist[k] != hist[k - 1]
        sparse = dense = 0
        for c0 in range(0, p, super_w):
            per_row = moved[:, c0:c0 + super_w].sum(axis=1)
            for r0 in range(0, q, tile):
                rows = per_row[r0:r0 + tile]
                if (rows > 0).sum() <= rows_max and rows.max() <= row_nz_max:
                    sparse += 1
                else:
                    dense += 1
        out.append((sparse, dense))
    return out


@pytest.mark.parametrize("q,p", [(512, 1024), (300, 777)])
def test_sparse_block_update(qe, oracle, q, p):
    """From the second sweep on, a block-update tile whose rows changed few
    codes applies only the nonzero code differences (QE_CD_DENSE turns this
    off).  Over 12 sweeps the run passes from dense to sparse tiles (checked
    from the codes); every sweep meets the parity bar against the oracle and
    leaves R = (What - W) Sigma to fp32 rounding, and the matrix-core-only
    run reaches the same objective."""
    W, X = layer(q, p, 2048, 43, corr=0.9)
    S32 = oracle.damp(oracle.gram(X), 0.01).astype(np.float32)
    scale, zero = oracle.grid_minmax(W, 4)
    sweeps = 12
    g = gpu_cd(qe, W, S32, 4, scale, zero, sweeps)
    regimes = block_update_regimes(g["hist"], q, p)
    print(f"{q}x{p}: (sparse, dense) block updates per sweep 2..{sweeps}: {regimes}")
    assert regimes[0][1] > 0                              # sweep 2: dense tiles
    assert sum(sp for sp, _ in regimes) > 0               # later: sparse tiles
    check_parity(oracle, W, S32, 4, scale, zero, g, f"sparse {q}x{p}")
    S64 = S32.astype(np.float64)
    for k in range(sweeps):
        D = g["whats"][k].astype(np.float64) - W
        bound = 1e-5 * (np.abs(D) @ np.abs(S64)) + 1e-30
        assert np.all(np.abs(g["Rs"][k] - D @ S64) <= bound), f"sweep {k + 1}"
    d = gpu_cd(qe, W, S32, 4, scale, zero, sweeps, extra=qe.QE_CD_DENSE)
    check_parity(oracle, W, S32, 4, scale, zero, d, f"dense {q}x{p}")
    assert d["obj"][-1] == pytest.approx(g["obj"][-1], rel=1e-6)


def test_on_grid_weights_bitwise(qe, oracle):
    q, p = 100, 230
    k = synth.integers((q, p), seed=20, lo=0, hi=16)
    scale = np.full(q, 2.0 ** -6, np.float32)
    zero = synth.integers((q,), seed=21, lo=0, hi=16).astype(np.float32)
    W = (scale[:, None] * (k - zero[:, None])).astype(np.float32)
    X = synth.correlated_activations(p, 512, 0.9, 22)
    S32 = oracle.damp(oracle.gram(X), 0.01).astype(np.float32)
    g = gpu_cd(qe, W, S32, 4, scale, zero, 3)
    assert np.array_equal(g["codes"], k)
    assert np.array_equal(g["What"], W)
    assert not np.any(g["R"])
    assert all(o == 0.0 for o in g["obj"])


def test_diagonal_sigma_is_round_to_nearest(qe, oracle):
    q, p = 64, 300
    W = synth.gaussian((q, p), seed=23, std=0.03)
    d = synth.uniform((p,), seed=24, lo=0.5, hi=3.0)
    S32 = np.diag(d).astype(np.float32)
    scale, zero = oracle.grid_minmax(W, 3)
    g = gpu_cd(qe, W, S32, 3, scale, zero, 3)
    ref = oracle.cd(W, S32, 3, scale, zero, 3)
    for k in range(3):
        assert np.array_equal(g["hist"][k], ref.codes_hist[k])


def test_tie_rule_fixture(qe, oracle):
    gd = json.load(open(os.path.join(GOLDEN, "cd_tie_rule.json")))
    W = np.array(gd["W"], np.float32)
    S32 = np.array(gd["Sigma"], np.float32)
    sc = np.array(gd["scale"], np.float32)
    ze = np.array(gd["zero"], np.float32)
    for case in gd["cases"]:
        if case["codes0"] is None:
            g = gpu_cd(qe, W, S32, gd["bits"], sc, ze, 1)
        else:
            c0 = np.array(case["codes0"], np.int32)
            W0 = oracle.dequant(c0, sc, ze).astype(np.float32)
            g = gpu_cd(qe, W, S32, gd["bits"], sc, ze, 1, W0=W0, codes0=c0)
        assert np.array_equal(g["codes"], case["expect"]), case


def test_hand_fixture(qe):
    gd = json.load(open(os.path.join(GOLDEN, "cd_two_by_two.json")))
    W = np.array(gd["W"], np.float32)
    S32 = np.array(gd["Sigma"], np.float32)
    g = gpu_cd(qe, W, S32, gd["bits"], np.array(gd["scale"], np.float32),
               np.array(gd["zero"], np.float32), gd["sweeps"])
    for k in range(gd["sweeps"]):
        assert np.array_equal(g["hist"][k], gd["codes_after_sweep"][k])
        assert g["obj"][k] == gd["f_after_sweep"][k]


@pytest.mark.parametrize("fp32", [False, True])
@pytest.mark.parametrize("q,p", [(120, 200), (256, 384)])
def test_warm_start_from_arbitrary_what(qe, oracle, q, p, fp32):
    # Sec. 3.1: CD may start from any What (e.g. another quantizer's output);
    # the residual is then formed by a full product (R = (What - W) Sigma)
    W, X = layer(q, p, 1024, 25, corr=0.9)
    S32 = oracle.damp(oracle.gram(X), 0.01).astype(np.float32)
    scale, zero = oracle.grid_minmax(W, 4)
    codes0 = np.clip(np.rint(W / scale[:, None] + zero[:, None]), 0, 15).astype(np.int32)
    W0 = oracle.dequant(codes0, scale, zero).astype(np.float32)
    g = gpu_cd(qe, W, S32, 4, scale, zero, 3, W0=W0, codes0=codes0,
               extra=qe.QE_CD_FP32 if fp32 else 0)
    compare_sweeps(oracle, W, S32, 4, scale, zero, g, f"warm start {q}x{p} fp32={fp32}", W0=W0,
                   codes0=codes0, codes_valid0=True)


def test_zero_diagonal_reports_error(qe):
    q, p = 8, 40
    W = synth.gaussian((q, p), seed=26)
    S = np.eye(p, dtype=np.float32)
    S[7, 7] = 0.0
    with pytest.raises(qe.QEError) as e:
        gpu_cd(qe, W, S, 4, np.ones(q, np.float32), np.zeros(q, np.float32), 1)
    assert e.value.code == 2


@pytest.mark.parametrize("q,p", [(140, 260), (256, 512), (512, 256)])
def test_objective_entry_point(qe, oracle, q, p):
    """Exact objective with and without H; q and p multiples of 256 take the
    256 x 256 tile kernels (one instantiation per set of present terms)."""
    W, X = layer(q, p, 1024, 27, corr=0.9)
    S32 = oracle.damp(oracle.gram(X), 0.01).astype(np.float32)
    scale, zero = oracle.grid_minmax(W, 4)
    g = gpu_cd(qe, W, S32, 4, scale, zero, 2)
    H = np.zeros_like(W)
    H.reshape(-1)[::97] = 0.01
    out = host(qe.objective(dev(W), dev(g["What"]), dev(S32), dev(H)))
    assert out[0] == pytest.approx(oracle.objective(W, g["What"], S32, H), rel=1e-5)
    assert out[1] == pytest.approx(oracle.objective(np.zeros_like(W), W, S32), rel=1e-5)
    out0 = host(qe.objective(dev(W), dev(g["What"]), dev(S32)))
    assert out0[0] == pytest.approx(g["obj"][-1], rel=1e-4)


def test_relaxed_sweeps_from_w_stay_at_w(qe, oracle):
    """From What = W with R = 0, a relaxed sweep writes beta = W exactly
    (Gauss-Seidel at its fixed point), so relaxed sweeps followed by the
    last, quantized sweep equal one plain sweep bitwise."""
    q, p = 96, 200
    W = synth.gaussian((q, p), seed=21, std=0.02)
    X = synth.correlated_activations(p, 1024, 0.9, 22)
    S32 = oracle.damp(oracle.gram(X), 0.01).astype(np.float32)
    scale, zero = oracle.grid_minmax(W, 4)
    out = []
    for sweeps, flags in ((3, qe.QE_INIT_FROM_W | qe.QE_RELAX_PERIOD(1)), (1, qe.QE_INIT_FROM_W)):
        Wd = dev(W)
        Wh = torch.empty_like(Wd)
        codes = torch.zeros((q, p), dtype=torch.uint8, device="cuda")
        R = torch.empty_like(Wd)
        qe.cd_sweep(Wd, dev(S32), 4, dev(scale), dev(zero), Wh, codes, R, sweeps, flags=flags)
        out.append((host(Wh), host(codes), host(R)))
    for a, b in zip(*out):
        assert np.array_equal(a, b)


@pytest.mark.parametrize("period,sweeps", [(2, 5), (3, 6)])
def test_relaxed_sweeps_match_oracle(qe, oracle, period, sweeps):
    q, p = 128, 257
    W = synth.gaussian((q, p), seed=23, std=0.02)
    X = synth.correlated_activations(p, 2048, 0.9, 24, out_channels=3, out_mult=20.0)
    S32 = oracle.damp(oracle.gram(X), 0.01).astype(np.float32)
    scale, zero = oracle.grid_minmax(W, 3)
    Wd = dev(W)
    Wh = torch.empty_like(Wd)
    codes = torch.zeros((q, p), dtype=torch.uint8, device="cuda")
    R = torch.empty_like(Wd)
    obj = torch.zeros(sweeps, dtype=torch.float64, device="cuda")
    qe.cd_sweep(Wd, dev(S32), 3, dev(scale), dev(zero), Wh, codes, R, sweeps,
                flags=qe.QE_INIT_FROM_W | qe.QE_RELAX_PERIOD(period), obj=obj)
    ref = oracle.cd(W, S32.astype(np.float64), 3, scale, zero, sweeps, relax_period=period)
    assert np.allclose(host(obj), ref.obj, rtol=1e-4)
    # the last sweep is quantized: codes agree (up to ties) and What is on the grid
    assert np.mean(host(codes).astype(np.int32) != ref.codes) <= 1e-3
    assert np.array_equal(host(Wh), oracle.dequant(host(codes), scale, zero).astype(np.float32))
    # R stays consistent with What through relaxed sweeps
    Rex = (host(Wh).astype(np.float64) - W) @ S32.astype(np.float64)
    assert np.max(np.abs(host(R) - Rex)) <= 1e-5 * np.max(np.abs(Rex)) + 1e-7


@pytest.mark.parametrize("where", ["W", "Sigma", "scale", "zero", "What", "R"])
def test_debug_checks_report_nonfinite_inputs(qe, oracle, where):
    """QE_DEBUG_CHECKS (footnote to Lemma 1: checks before the sweeps): a NaN
    or infinity in any input of the call is reported as QE_ERR_NONFINITE and
    the outputs are left as they were."""
    q, p, bits = 64, 160, 4
    W, X = layer(q, p, 512, 31, corr=0.9)
    S32 = oracle.damp(oracle.gram(X), 0.01).astype(np.float32)
    scale, zero = oracle.grid_minmax(W, bits)
    arrays = {"W": W.copy(), "Sigma": S32.copy(), "scale": scale.copy(), "zero": zero.copy()}
    # a warm start from What with a valid R: both are inputs then
    g = gpu_cd(qe, W, S32, bits, scale, zero, 1, per_sweep=False)
    arrays["What"], arrays["R"] = g["What"].copy(), g["R"].copy()
    a = arrays[where].reshape(-1)
    a[a.size // 3] = np.nan if where in ("W", "What", "zero") else np.inf
    Wd, Sd = dev(arrays["W"]), dev(arrays["Sigma"])
    Wh, R = dev(arrays["What"]), dev(arrays["R"])
    codes = dev(g["codes"].astype(np.uint8))
    before = (host(Wh).copy(), host(R).copy())
    flags = qe.QE_R_VALID | qe.QE_CODES_VALID | qe.QE_DEBUG_CHECKS
    with pytest.raises(qe.QEError) as e:
        qe.cd_sweep(Wd, Sd, bits, dev(arrays["scale"]), dev(arrays["zero"]), Wh, codes, R, 2,
                    flags=flags)
    assert e.value.code == qe.QE_ERR_NONFINITE
    assert np.array_equal(host(Wh), before[0], equal_nan=True)
    assert np.array_equal(host(R), before[1], equal_nan=True)


def test_debug_checks_pass_clean_inputs_unchanged(qe, oracle):
    """On finite inputs the flag changes nothing (bitwise), and an output-only
    What (QE_INIT_FROM_W) is not scanned even when it holds NaNs."""
    q, p, bits = 96, 250, 4
    W, X = layer(q, p, 1024, 32, corr=0.9)
    S32 = oracle.damp(oracle.gram(X), 0.01).astype(np.float32)
    scale, zero = oracle.grid_minmax(W, bits)
    out = []
    for flags in (qe.QE_INIT_FROM_W, qe.QE_INIT_FROM_W | qe.QE_DEBUG_CHECKS):
        Wd = dev(W)
        Wh = torch.full_like(Wd, float("nan"))
        R = torch.full_like(Wd, float("nan"))
        codes = torch.zeros((q, p), dtype=torch.uint8, device="cuda")
        obj = torch.zeros(3, dtype=torch.float64, device="cuda")
        qe.cd_sweep(Wd, dev(S32), bits, dev(scale), dev(zero), Wh, codes, R, 3, flags=flags,
                    obj=obj)
        out.append((host(Wh), host(codes), host(R), host(obj)))
    for x, y in zip(*out):
        assert np.array_equal(x, y)
