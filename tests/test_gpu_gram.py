"""GPU parity of qe_gram (Sigma = X X^T, Lemma 1) against the fp64 oracle.

Bar: relative Frobenius error <= 1e-5; Sigma exactly symmetric.  Every
product path is covered: the default split (on the 256 x 256 tiles the
two-way fp16 split of power-of-two-scaled channels, elsewhere the three-way
bf16 split), QE_GRAM_BF16X3 (the bf16 split on every tile) and QE_GRAM_FP32.
Tiles: p a multiple of 256 with n a multiple of 32 takes the 256 x 256
tiles, p a multiple of 128 the unguarded 128 x 128 loop, other shapes the
guarded one."""
import numpy as np
import pytest
import torch

import synth
from parity import dev, host, rel_fro

pytestmark = pytest.mark.gpu


def _gram(qe, X, layout=0, mode="default", **kw):
    return host(qe.gram(dev(X), layout=layout, fp32=mode == "fp32", bf16x3=mode == "bf16x3", **kw))


MODES = ["default", "bf16x3", "fp32"]


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("p,n", [(512, 2048), (200, 1000), (1, 7), (129, 33), (300, 5000),
                                 (384, 4096 + 32), (256, 16), (768, 4096 + 64),
                                 (256, 4096), (512, 8192 + 32)])
def test_gram_matches_oracle(qe, oracle, p, n, mode):
    """(256, 4096) takes 128 token splits of 32: the shortest K loop of the
    256 x 256 tile (two stages); (512, 8224) a split count that leaves a
    shorter last split."""
    spec = synth.CONFIGS["c1"]
    X = synth.activations(spec, n=n, p=p)
    S = _gram(qe, X, mode=mode)
    ref = oracle.gram(X)
    assert rel_fro(S, ref) <= 1e-5
    assert np.array_equal(S, S.T)


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("p,n", [(256, 1024), (130, 77), (384, 96), (512, 2048 + 17), (256, 31)])
def test_gram_token_major_layout(qe, oracle, p, n, mode):
    """(256, 1024) takes the 256 x 256 tiles; (512, 2065) an aligned part on
    them plus a 17-token tail; the others the 128 x 128 tiles."""
    X = synth.gaussian((p, n), seed=3)
    S_pn = _gram(qe, X, 0, mode=mode)
    S_np = _gram(qe, np.ascontiguousarray(X.T), 1, mode=mode)
    ref = oracle.gram(X)
    assert rel_fro(S_np, ref) <= 1e-5
    assert rel_fro(S_np, S_pn) <= 1e-6
    assert np.array_equal(S_np, S_np.T)


@pytest.mark.parametrize("layout", [0, 1])
def test_gram_split_products_exact_on_short_values(qe, layout):
    """Integers |x| <= 15 are their own bf16 h part (m = l = 0) and, scaled by
    the channel's power of two, their own fp16 h part (m = 0); with integer
    products and partial sums below 2^24 every step is exact (the scaling
    moves only exponents), so every product path returns the exact integer
    Gram."""
    rng = np.random.default_rng(11)
    X = rng.integers(-15, 16, size=(256, 2048)).astype(np.float32)
    exact = (X.astype(np.int64) @ X.T.astype(np.int64)).astype(np.float32)
    Xl = X if layout == 0 else np.ascontiguousarray(X.T)
    for mode in MODES:
        assert np.array_equal(_gram(qe, Xl, layout, mode=mode), exact), mode


@pytest.mark.parametrize("mode", ["default", "bf16x3"])
def test_gram_split_reconstructs_low_bits(qe, oracle, mode):
    """x = +-(1 + k 2^-20), k < 16: bf16(x) = +-1 and, with the channel
    scaled to 2^14 (1 + k 2^-20), fp16 of it is +-2^14, so all of the k part
    lives in the m plane of either split.  The off-diagonal error must stay
    far below what the h plane alone would give (the Gram of the signs)."""
    rng = np.random.default_rng(12)
    k = rng.integers(0, 16, size=(256, 512)).astype(np.float64)
    sgn = rng.choice([-1.0, 1.0], size=(256, 512))
    X = (sgn * (1.0 + k * 2.0 ** -20)).astype(np.float32)
    ref = oracle.gram(X)
    off = ~np.eye(256, dtype=bool)
    err = np.max(np.abs(_gram(qe, X, mode=mode) - ref)[off])
    gap = np.max(np.abs(oracle.gram(sgn.astype(np.float32)) - ref)[off])
    assert err <= 0.05 * gap


def _ranged_channels(p, n, seed):
    """Channels whose magnitudes span 2^-40 .. 2^40 (fp16 alone covers 2^-24
    .. 2^16), with special channels: all zero, a single nonzero, a largest
    |x| that is exactly a power of two, one just below a power of two (its
    scaled value rounds up to 2^15 in fp16), and values spread log-uniformly
    over 2^-30 .. 1 of the channel's largest."""
    rng = np.random.default_rng(seed)
    X = rng.standard_t(4, size=(p, n))
    X *= 2.0 ** rng.uniform(-40, 40, size=(p, 1))
    X[3] = 0.0
    X[5] = 0.0
    X[5, n // 3] = -3.0e-7
    X[7] = np.clip(X[7], -1.0, 1.0) * 2.0 ** 9
    X[7, 11] = 2.0 ** 10
    X[9] = np.clip(X[9], -1.0, 1.0)
    X[9, 17] = -np.float32(1 - 2.0 ** -24) * 2.0 ** 6
    X[11] = rng.choice([-1.0, 1.0], size=n) * 2.0 ** rng.uniform(-30, 0, size=n)
    return X.astype(np.float32)


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("layout", [0, 1])
def test_gram_tiny_elements_beside_a_large_one(qe, oracle, mode, layout):
    """Channel a holds one value 1 (its scale: 2^14 after scaling) and values
    2^-26 .. 2^-34 elsewhere, whose scaled h parts are fp16 subnormals; channel
    b is 0 where a is 1, so Sigma_ab comes from a's tiny values alone.  Their
    split keeps an absolute error of at most 2^-25 in scaled units (2^-39 of
    the channel's largest), a relative 2^-15 .. 2^-7 of each value, errors
    that average out over the tokens: Sigma_ab within 2e-3 of the oracle (a
    CPU model of the split gives 6e-4).  fp16 subnormals taken as 0 in the
    split would leave it off by about 18%."""
    p, n = 256, 2048
    rng = np.random.default_rng(31)
    X = rng.standard_normal((p, n))
    a, b = 1, 2
    X[a] = rng.choice([-1.0, 1.0], size=n) * 2.0 ** rng.uniform(-34, -26, size=n)
    X[a, 0] = 1.0
    X[b, 0] = 0.0
    X = X.astype(np.float32)
    Xl = X if layout == 0 else np.ascontiguousarray(X.T)
    S = _gram(qe, Xl, layout, mode=mode).astype(np.float64)
    ref = oracle.gram(X)
    assert abs(S[a, b] - ref[a, b]) <= 2e-3 * abs(ref[a, b])
    d = np.sqrt(np.diag(ref))
    assert np.all(np.abs(S - ref) <= 1e-5 * np.outer(d, d))


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("layout", [0, 1])
def test_gram_channel_scales(qe, oracle, mode, layout):
    """Every entry against the oracle relative to its Cauchy-Schwarz scale,
    |S_ij - ref_ij| <= 1e-5 sqrt(ref_ii ref_jj), on channels 2^80 apart (no
    single fp16 scale holds them, so this pins the per-channel power-of-two
    scaling and its exact removal); the all-zero channel's row and column
    exactly 0."""
    p, n = 256, 1024
    X = _ranged_channels(p, n, seed=21)
    Xl = X if layout == 0 else np.ascontiguousarray(X.T)
    S = _gram(qe, Xl, layout, mode=mode).astype(np.float64)
    ref = oracle.gram(X)
    d = np.sqrt(np.diag(ref))
    assert np.all(np.abs(S - ref) <= 1e-5 * np.outer(d, d))
    assert not np.any(S[3]) and not np.any(S[:, 3])
    assert np.array_equal(S, S.T)


@pytest.mark.parametrize("p,cuts", [(320, (1000, 2100)), (512, (1024, 2048 + 512))])
def test_gram_accumulates_token_chunks(qe, oracle, p, cuts):
    X = synth.gaussian((p, 3000 if p == 320 else 4096), seed=4)
    a, b = cuts
    Sigma = torch.empty((p, p), dtype=torch.float32, device="cuda")
    qe.gram(dev(X[:, :a]), Sigma=Sigma)
    qe.gram(dev(X[:, a:b]), Sigma=Sigma, accumulate=True)
    qe.gram(dev(X[:, b:]), Sigma=Sigma, accumulate=True, damp=0.01)
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


@pytest.mark.timeout(600)
@pytest.mark.parametrize("mode", ["default", "bf16x3"])
@pytest.mark.parametrize("layout,n", [(1, 2048 + 17), (0, 2048 + 32)])
def test_gram_direct_mode_large_p(qe, oracle, layout, n, mode):
    """33024 channels: the split partials of 33411 128 x 128 tiles would
    exceed the 2 GB budget, so each call writes Sigma directly (256 x 256
    tiles, the fp16 split or, with QE_GRAM_BF16X3, the bf16 one); token-major
    with a 17-token tail on the 128 x 128 tiles.  A seeded block of 256
    channels and every diagonal entry against the oracle's fp64 sums of the
    same numbers; the block exactly symmetric."""
    p = 33024
    ws = qe.load().qe_gram_workspace_size(p, n)
    assert ws < (64 << 20)                       # no split partials: direct mode
    rng = np.random.default_rng(41)
    X = rng.standard_t(4, size=(p, n)).astype(np.float32)
    X[rng.choice(p, 300, replace=False)] *= 30.0
    idx = np.sort(rng.choice(p, 256, replace=False))
    Xl = X if layout == 0 else np.ascontiguousarray(X.T)
    S = qe.gram(dev(Xl), layout=layout, bf16x3=mode == "bf16x3")
    idx_d = torch.as_tensor(idx, device="cuda")
    block = host(S[idx_d][:, idx_d])
    blockT = host(S[:, idx_d][idx_d])
    diag = host(torch.diagonal(S)).astype(np.float64)
    del S
    torch.cuda.empty_cache()
    ref_block = oracle.gram(X[idx])
    ref_diag = np.einsum("ij,ij->i", X.astype(np.float64), X.astype(np.float64))
    assert np.array_equal(block, blockT.T)
    assert rel_fro(block, ref_block) <= 1e-5
    assert np.max(np.abs(diag - ref_diag) / ref_diag) <= 1e-5
