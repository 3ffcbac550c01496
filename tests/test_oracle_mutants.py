"""The oracle's pins catch plausible mistakes (CPU only).

Each case plants one mistake in a private copy of the oracle -- the C source
compiled into a temporary library, or the Python module loaded from altered
text -- and runs the pin that should catch it against the broken copy; the
pin must fail.  The oracle's own files are never modified.  This backs the
claim that the pins are tight: a dropped term, a flipped sign, a wrong index,
a lost tie rule or a transposed operand anywhere in the oracle fails a pin.
"""
import importlib.util
import os
import subprocess
import sys
import tempfile

import pytest

import oracle as real_oracle
import test_oracle_basics as basics
import test_oracle_cd as cdpins
import test_oracle_outlier as outpins

ORACLE_DIR = os.path.dirname(real_oracle.__file__)
C_SRC = os.path.join(ORACLE_DIR, "qe_oracle.c")
PY_SRC = os.path.join(ORACLE_DIR, "__init__.py")


def _brute(o):
    cdpins.test_cd_equals_brute_force_coordinate_minimisation(o, 2, 0.9, 2)


def _brute_3bit(o):
    cdpins.test_cd_equals_brute_force_coordinate_minimisation(o, 3, 0.9, 3)


def _three_forms(o):
    cdpins.test_three_forms_agree(o, 0.9)


def _tie_fixture(o):
    cdpins.test_tie_rule_fixture(o)


def _grid_hand(o):
    basics.test_grid_hand_example(o)


def _gram_blas(o):
    basics.test_gram_matches_blas_product(o, 0)


def _gram_entries(o):
    basics.test_gram_entries_equal_full(o)


def _topk_lexsort(o):
    for s in (7, 50, 400, 1000):
        outpins.test_topk_matches_lexsort(o, s)
    outpins.test_topk_budget_cuts_a_tie_group(o)


def _iht_descent(o):
    outpins.test_iht_step_descends(o, 5)


def _identity_sigma(o):
    outpins.test_identity_sigma_closed_form(o)
    outpins.test_identity_sigma_step_size(o)


def _objective_direct(o):
    basics.test_objective_through_sigma_equals_direct(o)


def _damp(o):
    basics.test_damp_closed_form(o)


def _codes_on_grid(o):
    cdpins.test_iterates_stay_on_the_grid(o)


# (name, original text, planted text, pin that must fail)
C_MUTANTS = [
    ("lemma1 keeps the k = j term",
     "if (l != j) c += Sj[l] * w[l];", "c += Sj[l] * w[l];", _brute),
    ("lemma1 sign of beta",
     "double beta = -(c - T[i * p + j]) / Sj[j];", "double beta = (c - T[i * p + j]) / Sj[j];",
     _brute),
    ("lemma1 sign of the zero point",
     "continue;\n            }\n            double t = beta / scale[i] + zero[i];",
     "continue;\n            }\n            double t = beta / scale[i] - zero[i];",
     _brute),
    ("lemma1 Sigma column of the wrong coordinate",
     "double* w = Wh + i * p;\n        for (int64_t j = j0; j < p; ++j) {\n            const double* Sj = S + j * p;",
     "double* w = Wh + i * p;\n        for (int64_t j = j0; j < p; ++j) {\n            const double* Sj = S + ((j + 1) % p) * p;",
     _brute),
    ("modified-CD rule dropped (equal-distance current code not kept)",
     "fabs(t - (double)code) <= fabs(t - (double)kk)", "fabs(t - (double)code) < fabs(t - (double)kk)",
     _tie_fixture),
    ("ties rounded away from zero instead of to even",
     "double k = nearbyint(t);", "double k = round(t);", _tie_fixture),
    ("upper clamp to the finite grid missing",
     "if (k > (double)maxq) k = (double)maxq;", "", _codes_on_grid),
    ("alg1 first rank-1 half with the wrong sign",
     "for (int64_t l = 0; l < p; ++l) m[l] -= old * Sj[l];",
     "for (int64_t l = 0; l < p; ++l) m[l] += old * Sj[l];", _three_forms),
    ("alg2 partial sum over the whole row",
     "for (int64_t l = 0; l <= j; ++l) part", "for (int64_t l = 0; l < p; ++l) part", _three_forms),
    ("alg2 column of dW updated with the wrong sign",
     "dW[i * p + j] -= Wh[i * p + j];", "dW[i * p + j] += Wh[i * p + j];", _three_forms),
    ("gram with one operand repeated",
     "acc += x_at(X, p, n, layout, a, t) * x_at(X, p, n, layout, b, t);",
     "acc += x_at(X, p, n, layout, a, t) * x_at(X, p, n, layout, a, t);", _gram_blas),
    ("gram entries transposed in token-major layout",
     "return layout == 0 ? (double)X[a * n + t] : (double)X[t * p + a];",
     "return layout == 0 ? (double)X[a * n + t] : (double)X[a * n + t];", _gram_entries),
    ("P_s ties to the higher index",
     "return (x->idx < y->idx) ? -1 : (x->idx > y->idx);",
     "return (x->idx > y->idx) ? -1 : (x->idx < y->idx);", _topk_lexsort),
    ("P_s counts exact zeros",
     "if (kv[r].key == 0.0) break;", "", _topk_lexsort),
    ("grid zero point not rounded",
     "zero[i] = rintf(negq);", "zero[i] = negq;", _grid_hand),
]

PY_MUTANTS = [
    ("alg2 diagonal zeroed before P is formed",
     "        P = _c(tgt @ N, np.float64)            # P = W Sigma^norm, before zeroing the diagonal\n"
     "        N = _c(N, np.float64)\n"
     "        N[np.diag_indices_from(N)] = 0.0       # then Sigma^norm_jj = 0\n",
     "        N = _c(N, np.float64)\n"
     "        N[np.diag_indices_from(N)] = 0.0\n"
     "        P = _c(tgt @ N, np.float64)\n",
     _three_forms),
    ("IHT step climbs the gradient",
     "V = H - eta * grad", "V = H + eta * grad", _iht_descent),
    ("IHT step size 1/lambda instead of 1/(2 lambda)",
     "eta = 1.0 / (2.0 * float(lam))", "eta = 1.0 / float(lam)", _identity_sigma),
    ("objective ignores H",
     "        D = D + np.asarray(H, np.float64)\n", "        D = D\n", _objective_direct),
    ("damping by the trace instead of the mean diagonal",
     "mean_diag = float(np.sum(np.diag(S))) / S.shape[0]", "mean_diag = float(np.sum(np.diag(S)))",
     _damp),
]


def _plant(text, old, new, name):
    assert text.count(old) == 1, f"{name}: the original text must occur exactly once"
    return text.replace(old, new)


def _run_pin_expecting_failure(pin, o, name):
    try:
        pin(o)
    except (AssertionError, ValueError):
        return
    pytest.fail(f"planted mistake '{name}' passed its pin {pin.__name__}")


@pytest.fixture(scope="module")
def tmpdir_mod():
    with tempfile.TemporaryDirectory(dir="/tmp") as d:
        yield d


@pytest.mark.parametrize("name,old,new,pin", C_MUTANTS, ids=[m[0] for m in C_MUTANTS])
def test_c_mutant_fails_its_pin(tmpdir_mod, name, old, new, pin):
    src = _plant(open(C_SRC).read(), old, new, name)
    tag = str(abs(hash(name)))
    c_path = os.path.join(tmpdir_mod, f"mutant_{tag}.c")
    so_path = os.path.join(tmpdir_mod, f"libmutant_{tag}.so")
    with open(c_path, "w") as f:
        f.write(src)
    subprocess.run(["gcc", "-O2", "-fopenmp", "-ffp-contract=off", "-std=c11", "-shared", "-fPIC",
                    "-w", "-o", so_path, c_path, "-lm"], check=True)
    real_oracle._load()
    saved = real_oracle._lib
    real_oracle._lib = real_oracle.bind(so_path)
    try:
        _run_pin_expecting_failure(pin, real_oracle, name)
    finally:
        real_oracle._lib = saved
    # the untouched oracle passes the same pin
    pin(real_oracle)


@pytest.mark.parametrize("name,old,new,pin", PY_MUTANTS, ids=[m[0] for m in PY_MUTANTS])
def test_python_mutant_fails_its_pin(name, old, new, pin):
    src = _plant(open(PY_SRC).read(), old, new, name)
    spec = importlib.util.spec_from_loader("oracle_mutant", loader=None)
    mod = importlib.util.module_from_spec(spec)
    mod.__file__ = PY_SRC            # the mutant binds the real C library
    sys.modules["oracle_mutant"] = mod
    try:
        exec(compile(src, "oracle_mutant", "exec"), mod.__dict__)
        _run_pin_expecting_failure(pin, mod, name)
    finally:
        del sys.modules["oracle_mutant"]
    pin(real_oracle)


def test_mutants_cover_every_oracle_function():
    """Every arithmetic routine of the C oracle carries at least one planted
    mistake above."""
    src = open(C_SRC).read()
    defs = ["static inline double x_at(", "void qeo_gram(", "void qeo_gram_entries(", "void qeo_grid_minmax(",
            "static int grid_decide(", "int qeo_cd_sweep_lemma1(", "int qeo_cd_sweep_alg1(",
            "void qeo_cd_sweep_alg2(", "static int kv_cmp(", "int64_t qeo_topk_abs("]
    starts = sorted((src.index(d), d) for d in defs)
    hits = {d: 0 for d in defs}
    for _, old, _, _ in C_MUTANTS:
        pos = src.index(old)
        hits[max(s for s in starts if s[0] < pos)[1]] += 1
    # qeo_gram_entries has no arithmetic of its own beyond x_at and the dot
    # product qeo_gram also has; both of those carry mutants
    assert not [d for d, h in hits.items() if h == 0 and d != "void qeo_gram_entries("], hits
