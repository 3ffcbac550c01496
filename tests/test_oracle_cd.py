"""Pins for the oracle's coordinate descent (Sec. 3).

What fixes the oracle here, other than the oracle itself:
* eq. (cd-highlevel) solved by brute force -- every grid value of a coordinate
  tried, f recomputed from X -- sweep by sweep on tiny layers;
* hand-derived fixtures under tests/golden/;
* Lemma 2 (convergence to a coordinate-wise minimum), checked by enumeration;
* exhaustive search over all (2^b)^p codes of a row (rows are independent):
  CD can never beat the optimum;
* monotone f after the first feasible iterate (Sec. 3.1);
* closed-form special cases: weights already on the grid, diagonal Sigma
  (round-to-nearest), exact ties, and unquantized sweeps (Gauss-Seidel on
  What Sigma = W Sigma, whose solution is What = W);
* the three written forms (Lemma 1 direct, Algorithm "QuantEase",
  Algorithm "Accelerated QuantEase") give the same iterates.
"""
import itertools
import json
import os

import numpy as np
import pytest

import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def f_from_x(W, Wh, X):
    return float(np.linalg.norm((np.asarray(W, np.float64) - np.asarray(Wh, np.float64))
                                @ np.asarray(X, np.float64)) ** 2)


def brute_force_sweeps(W, X, scale, zero, bits, sweeps):
    """Cyclic CD straight from eq. (cd-highlevel): for each (i, j) in order,
    try every level of Q_i, recompute f from X, keep the best (the current
    value unless another is strictly better)."""
    Wh = np.asarray(W, np.float64).copy()
    q, p = Wh.shape
    levels = [scale[i] * (np.arange(2 ** bits, dtype=np.float64) - zero[i]) for i in range(q)]
    codes = np.full((q, p), -1, np.int64)
    hist = []
    for _ in range(sweeps):
        for j in range(p):
            for i in range(q):
                fs = []
                for v in levels[i]:
                    Wt = Wh.copy()
                    Wt[i, j] = v
                    fs.append(f_from_x(W, Wt, X))
                fs = np.array(fs)
                k = int(np.argmin(fs))
                if codes[i, j] >= 0 and not fs[k] < fs[codes[i, j]]:
                    k = int(codes[i, j])
                codes[i, j] = k
                Wh[i, j] = levels[i][k]
        hist.append(codes.copy())
    return Wh, codes, hist


def small_layer(q, p, n, seed, corr=0.0, bits=3):
    W = synth.gaussian((q, p), seed=seed, std=0.05)
    if corr > 0:
        X = synth.correlated_activations(p, n, corr, seed)
    else:
        X = synth.gaussian((p, n), seed=seed + 1000)
    return W, X


@pytest.mark.parametrize("seed,corr,bits", [(1, 0.0, 2), (2, 0.9, 2), (3, 0.9, 3), (4, 0.5, 1)])
def test_cd_equals_brute_force_coordinate_minimisation(oracle, seed, corr, bits):
    W, X = small_layer(3, 6, 24, seed, corr)
    S = oracle.gram(X)                     # undamped: f through Sigma equals ||(W - What) X||^2
    scale, zero = oracle.grid_minmax(W, bits)
    res = oracle.cd(W, S, bits, scale, zero, 4)
    Wb, cb, hist = brute_force_sweeps(W, X, scale.astype(np.float64), zero.astype(np.float64), bits, 4)
    for k in range(4):
        assert np.array_equal(res.codes_hist[k], hist[k]), f"sweep {k + 1}"
    assert np.allclose(res.What, Wb, rtol=0, atol=1e-15)
    assert res.obj[-1] == pytest.approx(f_from_x(W, Wb, X), rel=1e-10)


def test_cd_hand_fixture(oracle):
    g = json.load(open(os.path.join(GOLDEN, "cd_two_by_two.json")))
    W = np.array(g["W"], np.float32)
    S = np.array(g["Sigma"])
    res = oracle.cd(W, S, g["bits"], np.array(g["scale"], np.float32),
                    np.array(g["zero"], np.float32), g["sweeps"])
    for k in range(g["sweeps"]):
        assert np.array_equal(res.codes_hist[k], g["codes_after_sweep"][k])
        assert np.array_equal(res.what_hist[k], g["what_after_sweep"][k])
        assert res.obj[k] == g["f_after_sweep"][k]
    # the fixture's exhaustive minimum
    best = min(oracle.objective(W, np.array([[a, b]]), S)
               for a in (-0.5, 0.0, 0.5, 1.0) for b in (-0.5, 0.0, 0.5, 1.0))
    assert best == g["f_min_exhaustive"]


def test_tie_rule_fixture(oracle):
    g = json.load(open(os.path.join(GOLDEN, "cd_tie_rule.json")))
    W = np.array(g["W"], np.float32)
    S = np.array(g["Sigma"])
    sc = np.array(g["scale"], np.float32)
    ze = np.array(g["zero"], np.float32)
    for case in g["cases"]:
        for form in ("lemma1", "alg1", "alg2"):
            if case["codes0"] is None:
                res = oracle.cd(W, S, g["bits"], sc, ze, 1, form=form)
            else:
                c0 = np.array(case["codes0"], np.int32)
                res = oracle.cd(W, S, g["bits"], sc, ze, 1, W0=oracle.dequant(c0, sc, ze),
                                codes0=c0, codes_valid=True, form=form)
            assert np.array_equal(res.codes, case["expect"]), (form, case)


@pytest.mark.parametrize("corr", [0.0, 0.9])
def test_three_forms_agree(oracle, corr):
    W, X = small_layer(40, 33, 96, 11, corr)
    S = oracle.damp(oracle.gram(X), 0.01)
    scale, zero = oracle.grid_minmax(W, 3)
    runs = {f: oracle.cd(W, S, 3, scale, zero, 5, form=f) for f in ("lemma1", "alg1", "alg2")}
    for f in ("alg1", "alg2"):
        for k in range(5):
            assert np.array_equal(runs[f].codes_hist[k], runs["lemma1"].codes_hist[k]), (f, k)
        assert np.allclose(runs[f].What, runs["lemma1"].What, rtol=0, atol=1e-14)
        assert np.allclose(runs[f].obj, runs["lemma1"].obj, rtol=1e-12)


@pytest.mark.parametrize("seed,corr", [(21, 0.0), (22, 0.9), (23, 0.95)])
def test_monotone_after_first_sweep(oracle, seed, corr):
    W, X = small_layer(30, 40, 120, seed, corr)
    S = oracle.damp(oracle.gram(X), 0.01)
    scale, zero = oracle.grid_minmax(W, 3)
    res = oracle.cd(W, S, 3, scale, zero, 12)
    for k in range(1, len(res.obj)):
        assert res.obj[k] <= res.obj[k - 1] * (1 + 1e-12), k


def test_converges_to_cw_minimum(oracle):
    W, X = small_layer(5, 9, 30, 31, 0.9)
    S = oracle.gram(X)
    bits = 2
    scale, zero = oracle.grid_minmax(W, bits)
    res = oracle.cd(W, S, bits, scale, zero, 200)
    last_change = max(k for k in range(len(res.codes_hist))
                      if k == 0 or not np.array_equal(res.codes_hist[k], res.codes_hist[k - 1]))
    assert last_change < 199                      # Lemma 2: the modified CD stops moving
    Wh = res.What
    f0 = f_from_x(W, Wh, X)
    for i in range(W.shape[0]):
        for j in range(W.shape[1]):
            for k in range(2 ** bits):
                Wt = Wh.copy()
                Wt[i, j] = scale[i] * (k - zero[i])
                assert f_from_x(W, Wt, X) >= f0 * (1 - 1e-12)


def test_cd_never_beats_row_optimum(oracle):
    W, X = small_layer(6, 5, 40, 41, 0.9)
    S = oracle.gram(X)
    bits = 2
    scale, zero = oracle.grid_minmax(W, bits)
    res = oracle.cd(W, S, bits, scale, zero, 25)
    equal = 0
    for i in range(W.shape[0]):
        levels = scale[i] * (np.arange(4) - zero[i])
        best = min(f_from_x(W[i:i + 1], np.array([c], np.float64), X)
                   for c in itertools.product(levels, repeat=W.shape[1]))
        fi = f_from_x(W[i:i + 1], res.What[i:i + 1], X)
        assert fi >= best * (1 - 1e-12)
        equal += fi <= best * (1 + 1e-12)
    assert equal >= 1          # CD finds the exact optimum on some of these tiny rows


def test_on_grid_weights_are_a_fixed_point(oracle):
    rng = synth.integers((20, 30), seed=5, lo=0, hi=16)
    scale = np.full(20, 2.0 ** -6, np.float32)
    zero = synth.integers((20,), seed=6, lo=0, hi=16).astype(np.float32)
    W = (scale[:, None] * (rng - zero[:, None])).astype(np.float32)
    X = synth.correlated_activations(30, 80, 0.9, 7)
    S = oracle.damp(oracle.gram(X), 0.01)
    res = oracle.cd(W, S, 4, scale, zero, 3)
    assert np.array_equal(res.codes, rng)
    assert np.array_equal(res.What, W.astype(np.float64))
    assert all(f == 0.0 for f in res.obj)


def test_iterates_stay_on_the_grid(oracle):
    """Problem (1) is feasible only on Q_i: after every quantized sweep each
    code lies in [0, 2^b - 1] and What equals its grid level, also when the
    grid is too narrow for W (half the min/max step), so that Lemma 1's
    minimiser often falls outside the grid and must be clamped to its end."""
    W, X = small_layer(12, 20, 60, 61, 0.9)
    S = oracle.damp(oracle.gram(X), 0.01)
    bits = 2
    scale, zero = oracle.grid_minmax(W, bits)
    scale = (scale * np.float32(0.5)).astype(np.float32)
    res = oracle.cd(W, S, bits, scale, zero, 3)
    t0 = W.astype(np.float64) / scale[:, None] + zero[:, None]
    assert np.any(t0 > 2 ** bits - 1) and np.any(t0 < 0)      # the clamp is exercised
    for k in range(3):
        c = res.codes_hist[k]
        assert c.min() >= 0 and c.max() <= 2 ** bits - 1
        assert np.array_equal(res.what_hist[k], oracle.dequant(c, scale, zero))


def test_sweep_from_a_start_column_is_the_tail_of_a_sweep(oracle):
    """A sweep begun at column j0 from a state whose first j0 columns already
    hold a full sweep's values finishes exactly as that full sweep does."""
    W, X = small_layer(9, 30, 90, 62, 0.9)
    S = oracle.damp(oracle.gram(X), 0.01)
    scale, zero = oracle.grid_minmax(W, 3)
    first = oracle.cd(W, S, 3, scale, zero, 1)
    full = oracle.cd(W, S, 3, scale, zero, 1, W0=first.What, codes0=first.codes, codes_valid=True)
    for j0 in (1, 13, 29):
        w0 = first.What.copy()
        c0 = first.codes.copy()
        w0[:, :j0] = full.What[:, :j0]
        c0[:, :j0] = full.codes[:, :j0]
        tail = oracle.cd(W, S, 3, scale, zero, 1, W0=w0, codes0=c0, codes_valid=True,
                         start_col=j0)
        assert np.array_equal(tail.codes, full.codes)
        assert np.array_equal(tail.What, full.What)
        assert np.all(np.isinf(tail.margin_hist[0][:, :0]))


def test_diagonal_sigma_is_round_to_nearest(oracle):
    W = synth.gaussian((25, 40), seed=8, std=0.03)
    d = synth.uniform((40,), seed=9, lo=0.5, hi=3.0).astype(np.float64)
    S = np.diag(d)
    scale, zero = oracle.grid_minmax(W, 3)
    res = oracle.cd(W, S, 3, scale, zero, 3)
    t = W.astype(np.float64) / scale[:, None].astype(np.float64) + zero[:, None]
    rtn = np.clip(np.rint(t), 0, 7)
    for k in range(3):
        assert np.array_equal(res.codes_hist[k], rtn)


def test_unquantized_sweeps_solve_normal_equations(oracle):
    # With every sweep left unquantized CD is Gauss-Seidel on What Sigma = W Sigma,
    # whose unique solution (Sigma positive definite) is What = W.
    W = synth.gaussian((6, 12), seed=10, std=0.05)
    X = synth.correlated_activations(12, 60, 0.7, 11)
    S = oracle.damp(oracle.gram(X), 0.05)
    lib = oracle._load()
    q, p = W.shape
    T = np.ascontiguousarray(W.astype(np.float64) @ S)
    Wh = np.zeros((q, p))
    codes = np.zeros((q, p), np.int32)
    valid = np.zeros((q, p), np.uint8)
    sc = np.ones(q)
    ze = np.zeros(q)
    for _ in range(300):
        lib.qeo_cd_sweep_lemma1(oracle._p(T, oracle._f64p), oracle._p(np.ascontiguousarray(S), oracle._f64p),
                                q, p, 4, oracle._p(sc, oracle._f64p), oracle._p(ze, oracle._f64p),
                                oracle._p(Wh, oracle._f64p), oracle._p(codes, oracle._i32p),
                                oracle._p(valid, oracle._u8p), None, 1, 0)
    assert np.allclose(Wh, W.astype(np.float64), rtol=0, atol=1e-10)


def test_relaxed_period_keeps_last_sweep_quantized(oracle):
    W, X = small_layer(10, 14, 50, 51, 0.9)
    S = oracle.damp(oracle.gram(X), 0.01)
    scale, zero = oracle.grid_minmax(W, 3)
    res = oracle.cd(W, S, 3, scale, zero, 6, relax_period=3)
    # sweep 3 is unquantized (off-grid), sweep 6 is the last and quantized
    on_grid = oracle.dequant(res.codes, scale, zero)
    assert not np.allclose(res.what_hist[2], oracle.dequant(res.codes_hist[2], scale, zero))
    assert np.array_equal(res.What, on_grid)


def test_zero_diagonal_is_rejected(oracle):
    S = np.eye(3)
    S[1, 1] = 0.0
    W = np.ones((2, 3), np.float32)
    with pytest.raises(ValueError):
        oracle.cd(W, S, 2, np.ones(2, np.float32), np.zeros(2, np.float32), 1)


def test_margin_is_distance_to_nearest_boundary(oracle):
    W = np.array([[0.125, -0.375, 0.3, 10.0]], np.float32)
    S = np.eye(4)
    sc = np.array([0.25], np.float32)
    ze = np.array([2.0], np.float32)
    res = oracle.cd(W, S, 2, sc, ze, 1)
    t = W[0].astype(np.float64) / 0.25 + 2.0        # [2.5, 0.5, 3.2, 42]
    want = [0.0, 0.0, abs(3.2 - 2.5), 42 - 2.5]
    assert np.allclose(res.margin_hist[0][0], want, atol=1e-6)
