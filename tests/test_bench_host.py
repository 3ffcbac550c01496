"""Host-side checks of bench.py (no GPU): argument handling and the traffic
summary reader."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_helpers_present():
    for name in ("log", "cpu_baseline", "outlier_bench", "measured_traffic", "kernel_source_hash",
                 "main"):
        assert callable(getattr(bench, name)), name


def test_traffic_reader_keys():
    t = bench.measured_traffic()
    assert set(t) <= set(bench.KERNEL_SOURCES)
    assert all(isinstance(v, int) and v > 0 for v in t.values())


def test_source_hash_stable():
    for k in bench.KERNEL_SOURCES:
        assert bench.kernel_source_hash(k) == bench.kernel_source_hash(k)
        assert len(bench.kernel_source_hash(k)) == 64


def test_more_than_one_gpu_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_cpu_baseline_small():
    """The oracle baseline on a tiny sample: the fields the bench line carries,
    including the single-thread sweep run in a child process."""
    import numpy as np
    import oracle
    import synth
    spec = synth.CONFIGS["c1"]
    X = synth.activations(spec)[:, :256]
    W = synth.weights(spec)
    sc, ze = oracle.grid_minmax(W, spec.bits)
    r = bench.cpu_baseline(spec, np.ascontiguousarray(X), W, sc, ze, spec.sweeps)
    assert r["kind"] == "oracle" and r["unit"] == "column-updates/s"
    assert r["value"] > 0 and r["cores"] >= 1 and r["cpu_model"]
    one = r["one_thread_sweep"]
    assert one["rows"] == min(bench.CPU_ONE_THREAD_ROWS, spec.q) and one["seconds"] > 0
    assert "256 of 2048 tokens" in r["sample"]
    assert r["value"] == spec.p / r["sweep_s"]
    full = bench.cpu_baseline(spec, np.ascontiguousarray(X), W[:64], sc[:64], ze[:64], 2,
                              full=True)
    assert "all 2 sweeps over all" in full["sample"]


def test_profile_readers():
    """The committed launch and parity records parse (or are absent)."""
    for rec in (bench.profiled_panel_launch(), bench.parity_record()):
        assert rec is None or isinstance(rec, dict)


def test_help_lists_the_switches():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--help"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 0
    for flag in ("--gpus", "--steps", "--warmup", "--no-cpu", "--no-outlier", "--no-peaks",
                 "--calib-copy", "--configs", "--oracle-sample"):
        assert flag in r.stdout, flag


def test_configs_report_rows(monkeypatch, tmp_path):
    """The per-configuration rows: the timings pass through; panel bandwidth
    and matrix-core busy come from the committed profile only while its
    source hash matches the step kernel's sources."""
    rep = {"configs": {"w": {"q": 4096, "p": 4096, "sweep_s": 1e-3}}}
    prof = tmp_path / "p.md"
    monkeypatch.setattr(bench, "CONFIG_PROFILE", str(prof))
    prof.write_text('```json\n{"source_sha256": "%s", "configs": {"w": '
                    '{"panel_only_launch_us": 26.0, "mfma_busy": 0.2}}}\n```\n'
                    % bench.kernel_source_hash("cd_step_kernel"))
    row = bench.configs_report(rep)["w"]
    assert row["sweep_s"] == 1e-3 and row["cd_step_mfma_busy"] == 0.2
    assert abs(row["panel"]["achieved_GBps"] - 17.0 * 4096 * 256 / 26e-6 / 1e9) < 1e-6
    prof.write_text('```json\n{"source_sha256": "0", "configs": {"w": '
                    '{"panel_only_launch_us": 26.0, "mfma_busy": 0.2}}}\n```\n')
    row = bench.configs_report(rep)["w"]
    assert row["panel"] is None and row["cd_step_mfma_busy"] is None
