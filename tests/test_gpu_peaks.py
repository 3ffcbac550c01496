"""Peak checks (libqe_peak.so) on the GPU: the measured matrix-core and copy
rates are positive, below the vendor peaks they are compared with, and the
copy is exact."""
import pytest

torch = pytest.importorskip("torch")


@pytest.mark.gpu
def test_measured_peaks_are_sane():
    from paper_2309_01885_amd import peaks
    m = peaks.measure(torch, bf16_iters=1000, f32_iters=500, copy_bytes=1 << 28)
    print(m, flush=True)
    assert m["copy_checked"]
    assert 0.3 * 2500 < m["mfma_bf16_tflops"] < 1.05 * 2500
    assert 0.3 * 2500 < m["mfma_f16_tflops"] < 1.05 * 2500
    assert 0.3 * 157.3 < m["mfma_f32_tflops"] < 1.05 * 157.3
    assert 0.5 < m["engine_clock_ghz_under_mfma"] < 2.6
    assert 0 < m["copy_gbps"] < 8000
