"""GPU parity of qe_gram (Sigma = X X^T, Lemma 1) against the fp64 oracle.

Bar: relative Frobenius error <= 1e-5; Sigma exactly symmetric."""
import numpy as np
import pytest
import torch

import synth
from parity import dev, host, rel_fro

pytestmark = pytest.mark.gpu


def _gram(qe, X, layout=0, **kw):
    return host(qe.gram(dev(X), layout=layout, **kw))


@pytest.mark.parametrize("p,n", [(512, 2048), (200, 1000), (1, 7), (129, 33), (300, 5000)])
def test_gram_matches_oracle(qe, oracle, p, n):
    spec = synth.CONFIGS["c1"]
    X = synth.activations(spec, n=n, p=p)
    S = _gram(qe, X)
    ref = oracle.gram(X)
    assert rel_fro(S, ref) <= 1e-5
    assert np.array_equal(S, S.T)


@pytest.mark.parametrize("p,n", [(256, 1024), (130, 77)])
def test_gram_token_major_layout(qe, oracle, p, n):
    X = synth.gaussian((p, n), seed=3)
    S_pn = _gram(qe, X, 0)
    S_np = _gram(qe, np.ascontiguousarray(X.T), 1)
    ref = oracle.gram(X)
    assert rel_fro(S_np, ref) <= 1e-5
    assert rel_fro(S_np, S_pn) <= 1e-6
    assert np.array_equal(S_np, S_np.T)


def test_gram_accumulates_token_chunks(qe, oracle):
    X = synth.gaussian((320, 3000), seed=4)
    Sigma = torch.empty((320, 320), dtype=torch.float32, device="cuda")
    qe.gram(dev(X[:, :1000]), Sigma=Sigma)
    qe.gram(dev(X[:, 1000:2100]), Sigma=Sigma, accumulate=True)
    qe.gram(dev(X[:, 2100:]), Sigma=Sigma, accumulate=True, damp=0.01)
    ref = oracle.damp(oracle.gram(X), 0.01)
    S = host(Sigma)
    assert rel_fro(S, ref) <= 1e-5
    assert np.array_equal(S, S.T)


def test_gram_damping(qe, oracle):
    X = synth.gaussian((96, 500), seed=5)
    S = _gram(qe, X, damp=0.01)
    ref = oracle.damp(oracle.gram(X), 0.01)
    assert rel_fro(S, ref) <= 1e-5
    assert np.allclose(np.diag(S), np.diag(ref), rtol=1e-5)


def test_gram_deterministic(qe):
    X = synth.gaussian((384, 4096), seed=6)
    a = _gram(qe, X)
    b = _gram(qe, X)
    assert np.array_equal(a, b)


def test_gram_heavy_tailed_with_outlier_channels(qe, oracle):
    # the paper's workload statistics at a size the oracle finishes quickly:
    # Student-t(4) tokens and 1% outlier channels x30
    spec = synth.CONFIGS["c2"]
    X = synth.activations(spec, n=4096, p=640)
    S = _gram(qe, X, damp=0.01)
    ref = oracle.damp(oracle.gram(X), 0.01)
    assert rel_fro(S, ref) <= 1e-5
