"""Comparison helpers shared by the GPU parity tests (no method arithmetic)."""
import numpy as np
import torch


def dev(a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype is not None:
        t = t.to(dtype)
    return t.cuda()


def host(t):
    return t.detach().cpu().numpy()


def rel_fro(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return float(np.linalg.norm(a - b) / np.linalg.norm(b))


def first_divergence(codes_gpu_hist, codes_ref_hist):
    """For each row, the (sweep, column) of the first code that differs
    between the two sweep histories, scanning sweeps in order and columns in
    order inside a sweep; None for rows that never differ."""
    q = codes_ref_hist[0].shape[0]
    out = [None] * q
    for k, (g, r) in enumerate(zip(codes_gpu_hist, codes_ref_hist)):
        diff = np.asarray(g) != np.asarray(r)
        for i in np.nonzero(diff.any(axis=1))[0]:
            if out[i] is None:
                out[i] = (k, int(np.argmax(diff[i])))
    return out


def check_row_sampled_sweeps(W_rows, S64, whats, Rs, codes_hist, ref, obj_rtol=1e-4,
                             tie_margin=1e-4, max_split_rate=1e-6):
    """Per-sweep comparison of a row sample against the oracle's replay.

    CD visits the coordinates of a row in a fixed order, so two correct runs
    share every code until one of them meets an exact tie of the grid
    distance and takes the other, equally near level; from there on both rows
    are valid but different CD paths (several results are correct).  So:
    rows that never split must hold identical codes after every sweep and
    their objective must agree within obj_rtol; every split must start at an
    oracle tie (margin <= tie_margin grid units); split rows must stay valid
    CD paths (their objective never increases); splits must be rare (fp32
    rounding of t reaches ~1e-6 grid units, so about one decision in a
    million sits that close to a tie: at most max(2, max_split_rate x the
    number of decisions) splits).  Returns the number of split rows."""
    W64 = np.asarray(W_rows, np.float64)
    splits = first_divergence(codes_hist, ref.codes_hist)
    same = np.array([d is None for d in splits])
    decisions = codes_hist[0].size * len(codes_hist)
    assert (~same).sum() <= max(2, max_split_rate * decisions), \
        f"{int((~same).sum())} of {len(same)} rows split over {decisions} decisions"
    f_prev = None
    for k in range(len(codes_hist)):
        f_gpu = np.sum((whats[k].astype(np.float64) - W64) * Rs[k], axis=1)
        D = ref.what_hist[k] - W64
        f_ref = np.sum((D @ S64) * D, axis=1)
        if same.any():
            assert np.array_equal(codes_hist[k][same], ref.codes_hist[k][same]), f"sweep {k + 1}"
            assert np.sum(f_gpu[same]) == pytest_approx(np.sum(f_ref[same]), obj_rtol), \
                f"sweep {k + 1}: objective over the {int(same.sum())} rows that never split"
        if f_prev is not None and not same.all():
            split_rows = ~same
            assert np.all(f_gpu[split_rows] <= f_prev[split_rows] * (1 + 1e-6) + 1e-9), \
                f"sweep {k + 1}: a split row's objective went up"
        f_prev = f_gpu
    for i, d in enumerate(splits):
        if d is not None:
            assert ref.margin_hist[d[0]][i, d[1]] <= tie_margin, \
                f"row {i} splits at sweep {d[0] + 1}, column {d[1]} away from a tie " \
                f"(margin {ref.margin_hist[d[0]][i, d[1]]:.3e})"
    return int((~same).sum())


def pytest_approx(value, rtol):
    import pytest
    return pytest.approx(value, rel=rtol)
