"""Pins for the oracle's Gram matrix, damping, grid and objective.

Each check compares the oracle against something other than itself: a
closed form, a hand-derived fixture, or a library routine computing the same
quantity by a different route (numpy's BLAS product against the oracle's
plain loops)."""
import json
import os

import numpy as np
import pytest

import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ---------------------------------------------------------------- Gram (Lemma 1)
@pytest.mark.parametrize("layout", [0, 1])
def test_gram_matches_blas_product(oracle, layout):
    X = synth.gaussian((37, 203), seed=1)
    Xin = X if layout == 0 else np.ascontiguousarray(X.T)
    S = oracle.gram(Xin, layout)
    ref = X.astype(np.float64) @ X.astype(np.float64).T
    assert np.allclose(S, ref, rtol=1e-13, atol=1e-10)
    assert np.array_equal(S, S.T)


@pytest.mark.parametrize("layout", [0, 1])
def test_gram_blas_equals_plain_loops(oracle, layout):
    X = synth.gaussian((45, 1000), seed=11)
    Xin = X if layout == 0 else np.ascontiguousarray(X.T)
    S = oracle.gram_blas(Xin, layout, chunk=96, row_block=16)   # ragged last chunk and block
    assert np.allclose(S, oracle.gram(Xin, layout), rtol=1e-13, atol=1e-11)
    S2 = oracle.gram_blas(Xin[:, :300] if layout == 0 else Xin[:300], layout)
    oracle.gram_blas(Xin[:, 300:] if layout == 0 else Xin[300:], layout, out=S2)
    assert np.allclose(S2, S, rtol=1e-13, atol=1e-11)


def test_gram_closed_forms(oracle):
    # rows of a Sylvester-Hadamard matrix are orthogonal: X X^T = n I
    H = np.array([[1.0]])
    for _ in range(4):
        H = np.block([[H, H], [H, -H]])
    S = oracle.gram(H.astype(np.float32))
    assert np.array_equal(S, 16.0 * np.eye(16))
    # all-ones X: every entry equals n
    S1 = oracle.gram(np.ones((5, 9), np.float32))
    assert np.array_equal(S1, np.full((5, 5), 9.0))


def test_gram_entries_equal_full(oracle):
    X = synth.gaussian((24, 77), seed=2)
    S = oracle.gram(X)
    ia = np.array([0, 3, 23, 5, 11])
    ib = np.array([0, 7, 23, 19, 2])
    e = oracle.gram_entries(X, ia, ib)
    assert np.allclose(e, S[ia, ib], rtol=1e-14, atol=0)
    eT = oracle.gram_entries(np.ascontiguousarray(X.T), ia, ib, layout=1)
    assert np.allclose(eT, e, rtol=1e-14, atol=0)


def test_damp_closed_form(oracle):
    S = np.diag([1.0, 2.0, 3.0])
    S[0, 2] = S[2, 0] = 0.5
    D = oracle.damp(S, 0.5)
    # mean of the diagonal is 2, so every diagonal entry grows by 1
    assert np.array_equal(np.diag(D), [2.0, 3.0, 4.0])
    assert D[0, 2] == 0.5 and D[2, 0] == 0.5
    assert np.array_equal(oracle.damp(S, 0.0), S)


# ---------------------------------------------------------------- grid
def test_grid_hand_example(oracle):
    g = json.load(open(os.path.join(GOLDEN, "grid_example.json")))
    W = np.array(g["W"], np.float32)
    H = np.array(g["H"], np.float32)
    # the exclusion mask only matters for the last row
    s, z = oracle.grid_minmax(W, g["bits"], H)
    want_s = np.array([np.float32(a) / np.float32(b) for a, b in g["scale_num_den"]], np.float32)
    assert np.array_equal(s, want_s)
    assert np.array_equal(z, np.array(g["zero"], np.float32))
    s0, z0 = oracle.grid_minmax(W[:4], g["bits"])
    assert np.array_equal(s0, want_s[:4]) and np.array_equal(z0, z[:4])


@pytest.mark.parametrize("bits", [2, 3, 4, 8])
def test_grid_properties(oracle, bits):
    W = synth.gaussian((64, 100), seed=3, std=0.02)
    W[5] = np.abs(W[5])          # all non-negative row
    W[6] = -np.abs(W[6])         # all non-positive row
    W[7] = 0.0                   # degenerate row
    s, z = oracle.grid_minmax(W, bits)
    maxq = 2 ** bits - 1
    assert np.all(s > 0)
    assert np.all(z == np.round(z)) and np.all(z >= 0) and np.all(z <= maxq)
    # zero is a grid level (k = z), and every weight lies within half a step of
    # the grid's range
    lo = s.astype(np.float64) * (0 - z)
    hi = s.astype(np.float64) * (maxq - z)
    assert np.all(W >= lo[:, None] - 0.5 * s[:, None] * (1 + 1e-5))
    assert np.all(W <= hi[:, None] + 0.5 * s[:, None] * (1 + 1e-5))
    # rows 5/6 pin the clamps of lo/hi at zero
    assert z[5] == 0 and z[6] == maxq


def test_grid_excludes_outliers(oracle):
    W = synth.gaussian((8, 50), seed=4, std=0.02)
    W[3, 10] = 1.0
    H = np.zeros_like(W)
    H[3, 10] = 1.0
    s_all, _ = oracle.grid_minmax(W, 3)
    s_ex, _ = oracle.grid_minmax(W, 3, H)
    assert s_ex[3] < s_all[3] / 5
    mask = np.ones(8, bool)
    mask[3] = False
    assert np.array_equal(s_ex[mask], s_all[mask])


# ---------------------------------------------------------------- objective
def test_objective_through_sigma_equals_direct(oracle):
    X = synth.gaussian((12, 40), seed=5)
    W = synth.gaussian((7, 12), seed=6)
    Wh = synth.gaussian((7, 12), seed=7)
    H = np.zeros_like(W)
    H[2, 3] = 0.7
    S = oracle.gram(X)
    direct = np.linalg.norm(W.astype(np.float64) @ X - (Wh.astype(np.float64) + H) @ X) ** 2
    assert oracle.objective(W, Wh, S, H) == pytest.approx(direct, rel=1e-12)
    relerr = oracle.rel_error(W, Wh, S)
    d2 = np.linalg.norm(W.astype(np.float64) @ X - Wh.astype(np.float64) @ X) ** 2
    assert relerr == pytest.approx(d2 / np.linalg.norm(W.astype(np.float64) @ X) ** 2, rel=1e-12)


# ---- export for serving (bit-packed codes, outliers as CSR)
def test_pack_codes_hand_fixture(oracle):
    # 4-bit: code j in the low nibble for even j; 3-bit: 8 codes per 3 bytes
    c4 = np.array([[1, 2, 3, 15, 0]])
    assert oracle.pack_codes(c4, 4).tolist() == [[0x21, 0xF3, 0x00]]
    c3 = np.array([[1, 2, 3, 4, 5, 6, 7, 0]])
    # bit stream (LSB first): 001 010 011 100 101 110 111 000 read little-endian per code
    assert oracle.pack_codes(c3, 3).tolist() == [[0b11010001, 0b01011000, 0b00011111]]


@pytest.mark.parametrize("bits", [1, 2, 3, 4, 5, 8])
def test_pack_roundtrip(oracle, bits):
    codes = synth.integers((7, 29), seed=bits, lo=0, hi=2 ** bits)
    packed = oracle.pack_codes(codes, bits)
    assert packed.shape == (7, (29 * bits + 7) // 8)
    assert np.array_equal(oracle.unpack_codes(packed, 29, bits), codes)


def test_outliers_csr_matches_scipy(oracle):
    import scipy.sparse as sp
    H = synth.gaussian((9, 13), seed=3)
    H[np.abs(H) < 1.2] = 0.0
    rowptr, cols, vals = oracle.outliers_csr(H, np.flatnonzero(H))
    ref = sp.csr_matrix(H)
    assert np.array_equal(rowptr, ref.indptr) and np.array_equal(cols, ref.indices)
    assert np.array_equal(vals, ref.data.astype(np.float32))
