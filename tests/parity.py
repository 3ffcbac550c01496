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
