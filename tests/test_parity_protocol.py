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


def test_protocol_explains_a_cascade_from_a_tie(oracle):
    """A GPU-like run that takes the other level at a constructed exact tie
    and follows the oracle's rule from there: every later difference in the
    row is traced back to that tie decision."""
    W, S, scale, zero, ref, hist, whats, Rs = _run(oracle, sweeps=1)
    i, j = 5, 3
    # move W_ij so that sweep 1 meets an exact tie at (i, j): with the other
    # columns fixed, t is affine in W_ij, so solve for t = m + 1/2 exactly
    t_of = lambda w: _t_at(oracle, W, S, scale, zero, i, j, w)
    a, b = t_of(0.0), t_of(1.0) - t_of(0.0)
    m = np.floor(t_of(float(W[i, j]))) + 0.5
    W2 = W.astype(np.float64).copy()
    W2[i, j] = (m - a) / b
    ref2 = oracle.cd(W2, S, 3, scale, zero, 1)
    assert ref2.margin_hist[0][i, j] <= 1e-9
    # the "GPU" takes the other neighbour at the tie, then continues exactly
    gpu = ref2.codes.copy()
    other = int(m - 0.5) if ref2.codes[i, j] == int(m + 0.5) else int(m + 0.5)
    w0 = W2.copy()
    c0 = np.zeros_like(gpu)
    w0[i, :j] = ref2.What[i, :j]
    c0[i, :j] = ref2.codes[i, :j]
    w0[i, j] = float(scale[i]) * (other - float(zero[i]))
    c0[i, j] = other
    tail = oracle.cd(W2[i:i + 1], S, 3, scale[i:i + 1], zero[i:i + 1], 1, W0=w0[i:i + 1],
                     codes0=c0[i:i + 1], start_col=j + 1)
    gpu[i] = tail.codes[0]
    whats = [oracle.dequant(gpu, scale, zero).astype(np.float32)]
    Rs = [(whats[0].astype(np.float64) - W2) @ S]
    stats = teacher_forced(oracle, W2, S, 3, scale, zero, [gpu], whats, Rs, code_frac=1.0)
    assert stats[0]["split_rows"] == 1
    (row, ties), = stats[0]["tie_decisions"]
    assert row == i and ties[0][0] == j
    # the objective is compared along the GPU's tie decision
    assert stats[0]["obj_rel_err"] <= 1e-8           # fp32 levels in whats and Rs
    assert stats[0]["obj_ref_along_ties"] == pytest.approx(
        oracle.objective(W2, whats[0], S), rel=1e-8)


def _t_at(oracle, W, S, scale, zero, i, j, w_ij):
    """Lemma 1's t at (i, j) in the first sweep from What = W, with W_ij = w_ij
    (read off the oracle's margin would lose the side; recomputed here from
    the oracle's state before column j)."""
    W2 = W.astype(np.float64).copy()
    W2[i, j] = w_ij
    part = oracle.cd(W2[i:i + 1], S, 3, scale[i:i + 1], zero[i:i + 1], 1)
    state = W2[i].copy()
    state[:j] = part.What[0, :j]
    c = sum(S[j, l] * state[l] for l in range(S.shape[0]) if l != j)
    beta = ((W2[i] @ S)[j] - c) / S[j, j]
    return beta / float(scale[i]) + float(zero[i])
