"""GPU parity of the serving export (bit-packed codes, outliers as CSR)
against the oracle's reference layout: integer and byte work, so bit-exact."""
import numpy as np
import pytest
import torch

import synth
from parity import dev, host

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("bits", [1, 2, 3, 4, 5, 7, 8])
@pytest.mark.parametrize("q,p", [(5, 29), (64, 4096), (3, 1)])
def test_pack_codes_bit_exact(qe, oracle, bits, q, p):
    codes = synth.integers((q, p), seed=bits * 10 + q, lo=0, hi=2 ** bits).astype(np.uint8)
    got = host(qe.pack_codes(dev(codes), bits))
    assert np.array_equal(got, oracle.pack_codes(codes, bits))


def test_outliers_csr_from_topk(qe, oracle):
    V = synth.gaussian((300, 257), seed=51)
    s = 2000
    out, sup, nnz = qe.topk_abs(dev(V), s)
    rowptr, cols, vals = qe.outliers_csr(out, sup, nnz)
    n = int(host(nnz)[0])
    ref_sup, ref_dense = oracle.topk_abs(V, s)
    r_rowptr, r_cols, r_vals = oracle.outliers_csr(ref_dense, ref_sup)
    assert np.array_equal(host(rowptr), r_rowptr)
    assert np.array_equal(host(cols)[:n], r_cols)
    assert np.array_equal(host(vals)[:n], r_vals)


def test_outliers_csr_empty(qe):
    H = torch.zeros((4, 6), dtype=torch.float32, device="cuda")
    sup = torch.zeros(3, dtype=torch.int64, device="cuda")
    nnz = torch.zeros(1, dtype=torch.int64, device="cuda")
    rowptr, _, _ = qe.outliers_csr(H, sup, nnz)
    assert not np.any(host(rowptr))
