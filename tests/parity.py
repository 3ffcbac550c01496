"""Comparison helpers shared by the GPU parity tests (no method arithmetic:
every number they compare comes from the HIP library or from the oracle).

CD parity protocol.  CD visits the coordinates of a row in a fixed order, so
two correct runs hold the same codes until one of them meets a tie of the
grid distance (Lemma 1's t half-way between two levels, to within the
rounding of the arithmetic) and takes the other, equally near level; from
there on both rows follow valid but different CD paths, and several results
are correct.  Two checks follow from that:

* ``teacher_forced`` (binding; the per-sweep bar).  For every sweep k the
  oracle runs that one sweep from the GPU's own state after sweep k - 1
  (What, codes; codes valid after the first sweep), so a divergence cannot
  carry over from one sweep to the next.  Asserted after every sweep, whether
  or not any row splits: at most 0.1% of the sample's codes differ from the
  oracle's; in every row the first differing code sits at an oracle tie
  (|frac(t) - 1/2| <= 1e-4 grid units), and every later difference in that
  row follows from tie decisions (the oracle, taking the GPU's level at each
  tie, reaches the GPU's codes); the GPU's objective over the sample agrees
  within 1e-4 relative with the oracle's along those same tie decisions.
* ``free_running`` (reported; partly asserted).  The oracle runs all sweeps
  on its own from the common start.  Asserted: each row's first divergence
  sits at an oracle tie; rows that never split agree on the objective within
  1e-4; split rows keep descending.  Reported: the fraction of differing
  codes after each sweep and the number of split rows.

With ``QE_PARITY_STATS`` set, both checks append their figures as one JSON
line to that file.
"""
import json
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import torch

OBJ_RTOL = 1e-4
CODE_FRAC = 1e-3
TIE_MARGIN = 1e-4


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


def log_stats(record):
    path = os.environ.get("QE_PARITY_STATS")
    if path:
        with open(path, "a") as f:
            f.write(json.dumps(record) + "\n")


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


def _obj_errors(rec, f_gpu, f_ref, f0, f_reported=None):
    """Objective errors of one sweep against the reference value f_ref, with
    the floor the fp32 storage of the levels sets: every What_ij is a level
    rounded to fp32 (relative error eps <= 2^-24, taken as 2^-23), which moves
    (W - What) X by at most eps ||W X|| and f = ||(W - What) X||^2 by at most
    2 eps sqrt(f ||W X||^2) + eps^2 ||W X||^2 (f0 = ||W X||_F^2)."""
    eps = 2.0 ** -23
    rec["obj_ref"] = f_ref
    rec["obj_atol"] = 2 * eps * np.sqrt(abs(f_ref) * f0) + eps * eps * f0
    rec["obj_abs_err"] = abs(f_gpu - f_ref)
    rec["obj_rel_err"] = rec["obj_abs_err"] / abs(f_ref) if f_ref else rec["obj_abs_err"]
    if f_reported is not None:
        rec["reported_obj_abs_err"] = abs(f_reported - f_ref)
        rec["reported_obj_rel_err"] = (rec["reported_obj_abs_err"] / abs(f_ref) if f_ref
                                       else rec["reported_obj_abs_err"])


def gpu_row_objective(W_rows, what, R):
    """f_i = <What_i - W_i, R_i> per row from the GPU's own residual (fp64 sum)."""
    return np.sum((np.asarray(what, np.float64) - np.asarray(W_rows, np.float64))
                  * np.asarray(R, np.float64), axis=1)


def explain_row(oracle, W_row, S64, bits, scale, zero, T_row, start_w, start_c, valid,
                gpu_codes, tie_margin=TIE_MARGIN, max_steps=64):
    """Follows one row of one sweep along the GPU's choices at ties.

    The oracle sweeps the row from the sweep's start state; at the first
    column where the GPU's code differs, that decision must be a tie (oracle
    margin <= tie_margin); the oracle then takes the GPU's code there and
    carries on from the next column (Lemma 1 from the same state), and so on
    to the end of the row.  Every code the GPU holds is thereby shown to be
    the oracle's, or a tie decision, or a consequence of earlier tie
    decisions.  Returns the list of (column, margin) of the tie decisions."""
    w = np.array(start_w, np.float64).reshape(1, -1)
    c = (np.zeros(w.shape, np.int32) if start_c is None
         else np.array(start_c, np.int32).reshape(1, -1))
    gpu_codes = np.asarray(gpu_codes).reshape(-1)
    level = scale.astype(np.float64) * (gpu_codes - zero.astype(np.float64))
    ties, j0 = [], 0
    for _ in range(max_steps):
        ref = oracle.cd(W_row, S64, bits, scale, zero, 1, W0=w, codes0=c, codes_valid=valid,
                        T=T_row, start_col=j0, with_obj=False)
        diff = np.nonzero(ref.codes[0, j0:] != gpu_codes[j0:])[0]
        if diff.size == 0:
            return ties
        j = j0 + int(diff[0])
        m = float(ref.margin_hist[0][0, j])
        assert m <= tie_margin, f"column {j}: the GPU's code differs at oracle margin {m:.3e} " \
            f"grid units (not a tie), after {len(ties)} tie decisions in this row"
        ties.append((j, m))
        # the state just after column j along the GPU's path
        w[0, :j + 1] = np.concatenate([ref.What[0, :j], level[j:j + 1]])
        c[0, :j + 1] = np.concatenate([ref.codes[0, :j], gpu_codes[j:j + 1]])
        j0 = j + 1
    raise AssertionError(f"more than {max_steps} tie decisions in one row")


def teacher_forced(oracle, W_rows, S64, bits, scale, zero, codes_hist, whats, Rs, *,
                   W0=None, codes0=None, codes_valid0=False, T=None, gpu_obj=None,
                   label="", obj_rtol=OBJ_RTOL, code_frac=CODE_FRAC, tie_margin=TIE_MARGIN,
                   explain=True):
    """Per-sweep teacher-forced comparison of a GPU run with the oracle.

    W_rows, scale, zero: the rows compared (all rows of the layer, or a
    seeded sample: rows are independent, so a sample is exact).  codes_hist,
    whats, Rs: the GPU's codes, What and R of those rows after each sweep.
    W0/codes0/codes_valid0: the state the GPU's first sweep started from
    (default: What = W, codes not valid).  gpu_obj: optional per-sweep
    objective the library reported for exactly these rows.  The objective is
    compared with the oracle's along the same path: in rows that split at a
    tie (every difference traced back to tie decisions by explain_row) the
    reference is the objective of the GPU's own levels, which the oracle
    reaches by taking the GPU's choice at each tie.  Returns the per-sweep
    figures."""
    W64 = np.asarray(W_rows, np.float64)
    if T is None:
        T = W64 @ S64
    f0 = float(np.sum(W64 * T))              # ||W X||_F^2 of the sample
    sweeps = len(codes_hist)
    stats = []
    for k in range(sweeps):
        if k == 0:
            start_w = W64 if W0 is None else np.asarray(W0, np.float64).reshape(W64.shape)
            start_c = None if codes0 is None else np.asarray(codes0, np.int32)
            valid = codes_valid0
        else:
            start_w = np.asarray(whats[k - 1], np.float64)
            start_c = np.asarray(codes_hist[k - 1], np.int32)
            valid = True
        ref = oracle.cd(W_rows, S64, bits, scale, zero, 1, W0=start_w, codes0=start_c,
                        codes_valid=valid, T=T)
        g = np.asarray(codes_hist[k])
        diff = g != ref.codes
        frac = float(diff.mean())
        split_rows = np.nonzero(diff.any(axis=1))[0]
        margins = [float(ref.margin_hist[0][i, int(np.argmax(diff[i]))]) for i in split_rows]
        f_ref = ref.obj[0]
        f_gpu = float(np.sum(gpu_row_objective(W_rows, whats[k], Rs[k])))
        rec = {"sweep": k + 1, "code_diff_frac": frac, "split_rows": int(len(split_rows)),
               "max_first_margin": max(margins) if margins else 0.0}
        _obj_errors(rec, f_gpu, f_ref, f0, None if gpu_obj is None else gpu_obj[k])
        rec["first_diff"] = [[int(i), int(np.argmax(diff[i])), m, int(diff[i].sum())]
                             for i, m in zip(split_rows, margins)]
        if explain:
            # every differing code of a split row traced back to tie decisions
            # (rows in parallel threads: the oracle's C loop releases the GIL)
            todo = [int(i) for i, m in zip(split_rows, margins) if m <= tie_margin]

            def one(i, start_w=start_w, start_c=start_c, valid=valid, g=g):
                return explain_row(oracle, W_rows[i:i + 1], S64, bits, scale[i:i + 1],
                                   zero[i:i + 1], T[i:i + 1], start_w[i],
                                   None if start_c is None else start_c[i], valid, g[i],
                                   tie_margin=tie_margin)

            with ThreadPoolExecutor(max(1, min(16, len(todo)))) as ex:
                found = list(ex.map(one, todo))
            rec["tie_decisions"] = [[i, [[j, mm] for j, mm in t]] for i, t in zip(todo, found)]
            if len(todo) and len(todo) == len(split_rows):
                # Along the GPU's tie decisions the oracle reaches exactly the
                # GPU's codes in every split row (explain_row), so the
                # reference objective of those rows is that of the GPU's
                # levels: compare the objective on the same path.
                rows = np.asarray(todo)
                lev = (np.asarray(scale, np.float64)[rows, None]
                       * (g[rows] - np.asarray(zero, np.float64)[rows, None]))
                d_ref = np.asarray(ref.What, np.float64)[rows] - W64[rows]
                d_gpu = lev - W64[rows]
                f_tie = (f_ref - float(np.sum(d_ref * (d_ref @ S64)))
                         + float(np.sum(d_gpu * (d_gpu @ S64))))
                rec["obj_ref_along_ties"] = f_tie
                _obj_errors(rec, f_gpu, f_tie, f0, None if gpu_obj is None else gpu_obj[k])
        stats.append(rec)
    log_stats({"check": "teacher_forced", "label": label, "rows": int(W64.shape[0]),
               "cols": int(W64.shape[1]), "sweeps": stats})
    for rec in stats:
        where = f"{label} sweep {rec['sweep']}"
        assert rec["code_diff_frac"] <= code_frac, \
            f"{where}: {rec['code_diff_frac']:.3e} of codes differ (teacher-forced)"
        for i, j, m, _ in rec["first_diff"]:
            assert m <= tie_margin, \
                f"{where}: row {i} first differs at column {j}, oracle margin {m:.3e} grid " \
                f"units (not a tie)"
        assert rec["obj_abs_err"] <= obj_rtol * abs(rec["obj_ref"]) + rec["obj_atol"], \
            f"{where}: objective (teacher-forced) off by {rec['obj_rel_err']:.3e}"
        if gpu_obj is not None:
            assert rec["reported_obj_abs_err"] <= obj_rtol * abs(rec["obj_ref"]) + rec["obj_atol"], \
                f"{where}: reported objective off by {rec['reported_obj_rel_err']:.3e}"
    return stats


def free_running(oracle, W_rows, S64, bits, scale, zero, codes_hist, whats, Rs, *, W0=None,
                 codes0=None, codes_valid0=False, T=None, label="", obj_rtol=OBJ_RTOL,
                 tie_margin=TIE_MARGIN):
    """End-to-end comparison: the oracle runs every sweep on its own from the
    common start.  Asserts what stays unique (first divergences at ties,
    identical rows agreeing on the objective, split rows descending) and
    returns the per-sweep code-difference fractions."""
    W64 = np.asarray(W_rows, np.float64)
    if T is None:
        T = W64 @ S64
    sweeps = len(codes_hist)
    ref = oracle.cd(W_rows, S64, bits, scale, zero, sweeps,
                    W0=None if W0 is None else np.asarray(W0, np.float64),
                    codes0=None if codes0 is None else np.asarray(codes0, np.int32),
                    codes_valid=codes_valid0, T=T)
    splits = first_divergence(codes_hist, ref.codes_hist)
    same = np.array([d is None for d in splits])
    fracs, f_prev = [], None
    for k in range(sweeps):
        fracs.append(float(np.mean(np.asarray(codes_hist[k]) != ref.codes_hist[k])))
        f_gpu = gpu_row_objective(W_rows, whats[k], Rs[k])
        D = ref.what_hist[k] - W64
        f_ref = np.sum((D @ S64) * D, axis=1)
        if same.any():
            a, b = float(np.sum(f_gpu[same])), float(np.sum(f_ref[same]))
            rec = {}
            _obj_errors(rec, a, b, float(np.sum((W64 * T)[same])))
            assert rec["obj_abs_err"] <= obj_rtol * abs(b) + rec["obj_atol"], \
                f"{label} sweep {k + 1}: objective over the {int(same.sum())} rows that never split"
        if f_prev is not None and not same.all():
            assert np.all(f_gpu[~same] <= f_prev[~same] * (1 + 1e-6) + 1e-12), \
                f"{label} sweep {k + 1}: a split row's objective went up"
        f_prev = f_gpu
    for i, d in enumerate(splits):
        if d is not None:
            m = ref.margin_hist[d[0]][i, d[1]]
            assert m <= tie_margin, \
                f"{label}: row {i} splits at sweep {d[0] + 1}, column {d[1]} away from a tie " \
                f"(margin {m:.3e})"
    rec = {"check": "free_running", "label": label, "rows": int(W64.shape[0]),
           "cols": int(W64.shape[1]), "split_rows": int((~same).sum()),
           "split_sweeps": sorted(int(d[0]) + 1 for d in splits if d is not None),
           "code_diff_frac": fracs}
    log_stats(rec)
    return rec
