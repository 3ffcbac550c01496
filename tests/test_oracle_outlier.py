"""Pins for the oracle's outlier-aware path (Sec. 4).

* P_s against an independent selection (numpy lexsort on (-|v|, index));
* Lemma 3: the IHT step never increases g (H sparse, ||H||_0 <= s);
* s = 0 reduces to the plain CD of Sec. 3;
* Sigma = c I: V = H - E/c = W - What in closed form, so H+ = P_s(W - What);
* lambda_max on a matrix with known eigenvalues (Householder-rotated diagonal);
* the initialisation H = P_s(W), What = W - H keeps What + H = W exactly.
"""
import numpy as np
import pytest

import synth


def lexsort_topk(v, s):
    v = np.asarray(v, np.float64).reshape(-1)
    order = np.lexsort((np.arange(v.size), -np.abs(v)))
    sel = [e for e in order[:s] if v[e] != 0.0]
    return np.sort(np.array(sel, np.int64))


@pytest.mark.parametrize("s", [0, 1, 7, 50, 400, 1000])
def test_topk_matches_lexsort(oracle, s):
    V = synth.gaussian((20, 30), seed=1)
    # inject exact ties in |v| and exact zeros
    V.reshape(-1)[::17] = 0.5
    V.reshape(-1)[5::23] = -0.5
    V.reshape(-1)[3::7] = 0.0
    sup, Hp = oracle.topk_abs(V, s)
    assert np.array_equal(sup, lexsort_topk(V, s))
    flat = Hp.reshape(-1)
    assert np.array_equal(flat[sup], V.reshape(-1)[sup])
    mask = np.ones(V.size, bool)
    mask[sup] = False
    assert np.all(flat[mask] == 0)


def test_topk_threshold_property(oracle):
    V = synth.gaussian((64, 64), seed=2)
    s = 300
    sup, _ = oracle.topk_abs(V, s)
    a = np.abs(V.reshape(-1))
    kept = a[sup]
    rest = np.delete(a, sup)
    assert len(sup) == s and kept.min() >= rest.max()


def _layer(q, p, n, seed, corr=0.9):
    W = synth.gaussian((q, p), seed=seed, std=0.05)
    W.reshape(-1)[::37] *= 8.0
    X = synth.correlated_activations(p, n, corr, seed)
    return W, X


def test_init_sums_to_w(oracle):
    W, _ = _layer(16, 20, 10, 3)
    sup, H, Wh = oracle.outlier_init(W, 12)
    assert len(sup) == 12
    assert np.array_equal(Wh + H, W.astype(np.float64))


def test_zero_budget_is_plain_cd(oracle):
    W, X = _layer(24, 30, 90, 4)
    S = oracle.damp(oracle.gram(X), 0.01)
    sc, ze = oracle.grid_minmax(W, 3)
    lam = oracle.lambda_max(S)
    r0 = oracle.outlier(W, S, 3, sc, ze, 0, lam, 4)
    rc = oracle.cd(W, S, 3, sc, ze, 4)
    assert np.array_equal(r0.codes, rc.codes)
    assert np.array_equal(r0.What, rc.What)
    assert np.allclose(r0.g, rc.obj, rtol=1e-12)
    assert not np.any(r0.H)


@pytest.mark.parametrize("seed", [5, 6])
def test_iht_step_descends(oracle, seed):
    W, X = _layer(30, 36, 100, seed)
    S = oracle.damp(oracle.gram(X), 0.01)
    s = int(0.02 * W.size)
    sup0, H0, _ = oracle.outlier_init(W, s)
    sc, ze = oracle.grid_minmax(W, 3, H0)
    lam = oracle.lambda_max(S)
    r = oracle.outlier(W, S, 3, sc, ze, s, lam, 6)
    for k in range(6):
        assert r.g[k] <= r.g_cd[k] * (1 + 1e-12), k          # Lemma 3
        if k > 0:
            assert r.g_cd[k] <= r.g[k - 1] * (1 + 1e-12), k  # CD step, H fixed
        assert len(r.support_hist[k]) <= s


def test_identity_sigma_closed_form(oracle):
    W, _ = _layer(12, 16, 10, 7)
    c = 2.5
    S = c * np.eye(16)
    s = 20
    sup0, H0, _ = oracle.outlier_init(W, s)
    sc, ze = oracle.grid_minmax(W, 3, H0)
    r = oracle.outlier(W, S, 3, sc, ze, s, c, 1)
    # with Sigma = c I the CD step is round-to-nearest of W - H0 ...
    t = (W.astype(np.float64) - H0) / sc[:, None].astype(np.float64) + ze[:, None]
    assert np.array_equal(r.codes, np.clip(np.rint(t), 0, 7))
    # ... and V = H - (What + H - W) c / c = W - What
    _, Hp = oracle.topk_abs(W.astype(np.float64) - r.What, s)
    assert np.array_equal(r.H, Hp)


def test_identity_sigma_step_size(oracle):
    """With Sigma = c I and eta = 1/(2c), V = H - eta 2 (What + H - W) c is
    W - What whatever H is.  The grid's zero point is moved half a step, so
    0 is not a level and every kept entry carries a rounding residue: a
    wrong step size then changes V's values on the support."""
    W, _ = _layer(12, 16, 10, 7)
    c = 4.0
    S = c * np.eye(16)
    s = 20
    sup0, H0, _ = oracle.outlier_init(W, s)
    sc, ze = oracle.grid_minmax(W, 3, H0)
    ze = (ze + np.float32(0.5)).astype(np.float32)
    r = oracle.outlier(W, S, 3, sc, ze, s, c, 1)
    V = W.astype(np.float64) - r.What
    sup, Hp = oracle.topk_abs(V, s)
    assert np.array_equal(r.support, sup)
    assert np.allclose(r.H, Hp, rtol=1e-12, atol=0)
    assert np.min(np.abs(r.What.reshape(-1)[sup])) > 0.25 * np.min(sc)


def test_topk_budget_cuts_a_tie_group(oracle):
    """The budget ends inside a group of equal |V|: the lower linear indices
    of the group are kept (ties: lower index first)."""
    V = synth.uniform((20, 30), seed=9, lo=-0.4, hi=0.4)
    V.reshape(-1)[::6] = 0.5             # 100 tied entries, alternating sign
    V.reshape(-1)[3::12] = -0.5
    V.reshape(-1)[1::60] = 1.0           # 10 entries above the group
    s = 60
    sup, _ = oracle.topk_abs(V, s)
    assert np.array_equal(sup, lexsort_topk(V, s))
    tied = np.nonzero(np.abs(V.reshape(-1)) == 0.5)[0]
    assert np.array_equal(np.intersect1d(sup, tied), tied[:s - 10])


def test_lambda_max_known_spectrum(oracle):
    p = 40
    lam = np.linspace(0.5, 7.25, p)
    v = synth.gaussian((p,), seed=8).astype(np.float64)
    v /= np.linalg.norm(v)
    Q = np.eye(p) - 2.0 * np.outer(v, v)        # Householder reflection: orthogonal
    S = Q @ np.diag(lam) @ Q.T
    assert oracle.lambda_max(S) == pytest.approx(7.25, rel=1e-13)


# ---- structured (column) outliers, Sec. 4.3 "Structured Outliers"
def lexsort_columns(V, c):
    V = np.asarray(V, np.float64)
    key = np.sum(V * V, axis=0).astype(np.float32)
    order = np.lexsort((np.arange(key.size), -key.astype(np.float64)))
    return np.sort(np.array([j for j in order[:c] if key[j] != 0.0], np.int64))


@pytest.mark.parametrize("c", [0, 1, 3, 7, 30])
def test_topk_columns_matches_lexsort(oracle, c):
    V = synth.gaussian((9, 24), seed=31)
    V[:, 5] = V[:, 2]            # equal norms: the lower column wins
    V[:, 11] = -V[:, 2]
    V[:, 7] = 0.0                # a zero column is never kept
    V[:, 19] = 0.0
    cols, sup, out = oracle.topk_columns(V, c)
    assert np.array_equal(cols, lexsort_columns(V, c))
    q, p = V.shape
    assert np.array_equal(sup, np.sort((np.arange(q)[:, None] * p + cols[None, :]).reshape(-1)))
    keep = np.zeros(p, bool)
    keep[cols] = True
    assert np.array_equal(out[:, keep], V[:, keep]) and not np.any(out[:, ~keep])


def test_topk_columns_is_the_projection(oracle):
    """Among all sets of c columns, the kept set leaves the smallest residual
    ||V - P(V)||_F (brute force over every subset)."""
    import itertools
    V = synth.gaussian((5, 7), seed=32)
    c = 3
    _, _, out = oracle.topk_columns(V, c)
    best = min(np.sum(np.delete(V, list(sub), axis=1).astype(np.float64) ** 2)
               for sub in itertools.combinations(range(7), c))
    assert np.sum((V - out).astype(np.float64) ** 2) == pytest.approx(best, rel=1e-12)


@pytest.mark.parametrize("seed", [8, 9])
def test_structured_iht_step_descends(oracle, seed):
    W, X = _layer(30, 36, 100, seed)
    S = oracle.damp(oracle.gram(X), 0.01)
    s = 4 * 30                   # 4 columns
    sup0, H0, _ = oracle.outlier_init(W, s, structured=True)
    assert len(sup0) == s and np.count_nonzero(np.any(H0 != 0, axis=0)) == 4
    sc, ze = oracle.grid_minmax(W, 3, H0)
    lam = oracle.lambda_max(S)
    r = oracle.outlier(W, S, 3, sc, ze, s, lam, 5, structured=True)
    for k in range(5):
        assert r.g[k] <= r.g_cd[k] * (1 + 1e-12), k          # Lemma 3 (exact projection)
        if k > 0:
            assert r.g_cd[k] <= r.g[k - 1] * (1 + 1e-12), k
        assert np.count_nonzero(np.any(r.H != 0, axis=0)) <= 4


def test_structured_identity_sigma_closed_form(oracle):
    W, _ = _layer(12, 16, 10, 10)
    c = 1.75
    S = c * np.eye(16)
    s = 3 * 12
    _, _, H0 = oracle.topk_columns(W.astype(np.float64), 3)
    sc, ze = oracle.grid_minmax(W, 3, H0)
    r = oracle.outlier(W, S, 3, sc, ze, s, c, 1, structured=True)
    _, _, Hp = oracle.topk_columns(W.astype(np.float64) - r.What, 3)
    assert np.array_equal(r.H, Hp)


def test_structured_budget_below_one_column_is_plain_cd(oracle):
    W, X = _layer(24, 30, 90, 11)
    S = oracle.damp(oracle.gram(X), 0.01)
    sc, ze = oracle.grid_minmax(W, 3)
    r0 = oracle.outlier(W, S, 3, sc, ze, 23, oracle.lambda_max(S), 3, structured=True)
    rc = oracle.cd(W, S, 3, sc, ze, 3)
    assert np.array_equal(r0.codes, rc.codes) and not np.any(r0.H)
