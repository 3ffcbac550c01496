"""CPU checks of the CD parity protocol itself (tests/parity.py).

A run of the oracle stands in for the GPU's run: the protocol must accept it,
and must reject it once a code is changed away from a tie, or once the
reported objective is off by more than the tolerance."""
import numpy as np
import pytest

import synth
from parity import free_running, teacher_forced


def _run(oracle, sweeps=4):
    W = synth.gaussian((40, 64), seed=71, std=0.02)
    X = synth.correlated_activations(64, 512, 0.9, 72)
    S = oracle.damp(oracle.gram(X), 0.01)
    scale, zero = oracle.grid_minmax(W, 3)
    ref = oracle.cd(W, S, 3, scale, zero, sweeps)
    whats = [w.astype(np.float32) for w in ref.what_hist]
    Rs = [(w.astype(np.float64) - W) @ S for w in whats]
    return W, S, scale, zero, ref, [c.copy() for c in ref.codes_hist], whats, Rs


def test_protocol_accepts_the_oracle_itself(oracle):
    W, S, scale, zero, ref, hist, whats, Rs = _run(oracle)
    tf = teacher_forced(oracle, W, S, 3, scale, zero, hist, whats, Rs, gpu_obj=ref.obj)
    assert all(r["code_diff_frac"] == 0.0 and r["split_rows"] == 0 for r in tf)
    fr = free_running(oracle, W, S, 3, scale, zero, hist, whats, Rs)
    assert fr["split_rows"] == 0 and max(fr["code_diff_frac"]) == 0.0


def test_protocol_rejects_a_code_away_from_a_tie(oracle):
    W, S, scale, zero, ref, hist, whats, Rs = _run(oracle)
    k, i = 2, 7
    j = int(np.argmax(ref.margin_hist[k][i]))        # the decision farthest from a tie
    hist[k][i, j] = (hist[k][i, j] + 1) % 8
    with pytest.raises(AssertionError, match="not a tie"):
        teacher_forced(oracle, W, S, 3, scale, zero, hist, whats, Rs)


def test_protocol_rejects_too_many_differing_codes(oracle):
    W, S, scale, zero, ref, hist, whats, Rs = _run(oracle)
    hist[1] = (hist[1] + 1) % 8
    with pytest.raises(AssertionError, match="of codes differ"):
        teacher_forced(oracle, W, S, 3, scale, zero, hist, whats, Rs)


def test_protocol_rejects_a_wrong_objective(oracle):
    W, S, scale, zero, ref, hist, whats, Rs = _run(oracle)
    Rs[3] = Rs[3] * (1 + 3e-4)
    with pytest.raises(AssertionError, match="objective"):
        teacher_forced(oracle, W, S, 3, scale, zero, hist, whats, Rs)
    obj = list(ref.obj)
    obj[0] *= 1 + 3e-4
    _, _, _, _, _, hist, whats, Rs = _run(oracle)
    with pytest.raises(AssertionError, match="reported objective"):
        teacher_forced(oracle, W, S, 3, scale, zero, hist, whats, Rs, gpu_obj=obj)
