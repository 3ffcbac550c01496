"""qe_cd_sweep_noalloc (the allocation-free variant of qe_cd_sweep) against
qe_cd_sweep, through the C ABI: two calls in a row, the second on a smaller
layer, each bit-identical to qe_cd_sweep on the same inputs (the same
kernels run on the library's fixed scratch instead of a workspace); the
status output reports a data error and is cleared by the next call.  The
call allocates nothing and enqueues only kernels, so it can be recorded in a
HIP graph (torch.cuda.CUDAGraph on the capturing stream): every replay, with
eager work and synchronisations between the replays, gives bitwise what the
eager call gives."""
import numpy as np
import pytest
import torch

import synth
from parity import dev, host

pytestmark = pytest.mark.gpu


def _layer(oracle, q, p, seed, bits):
    W = synth.gaussian((q, p), seed=seed, std=0.02)
    X = synth.correlated_activations(p, 1024, 0.9, seed, out_channels=max(1, p // 50),
                                     out_mult=20.0)
    S32 = oracle.damp(oracle.gram(X), 0.01).astype(np.float32)
    scale, zero = oracle.grid_minmax(W, bits)
    return W, S32, scale, zero


def _both(qe, W, S32, scale, zero, bits, sweeps, block):
    q, p = W.shape
    out = []
    for noalloc in (False, True):
        Wd, Sd = dev(W), dev(S32)
        Wh = torch.empty_like(Wd)
        codes = torch.zeros((q, p), dtype=torch.uint8, device="cuda")
        R = torch.empty_like(Wd)
        obj = torch.zeros(sweeps, dtype=torch.float64, device="cuda")
        status = torch.full((1,), -1, dtype=torch.int32, device="cuda")
        if noalloc:
            qe.cd_sweep_noalloc(Wd, Sd, bits, dev(scale), dev(zero), Wh, codes, R, sweeps,
                                block=block, obj=obj, status=status)
        else:
            qe.cd_sweep(Wd, Sd, bits, dev(scale), dev(zero), Wh, codes, R, sweeps, block=block,
                        obj=obj)
        torch.cuda.synchronize()
        out.append((host(Wh), host(codes), host(R), host(obj), int(host(status)[0])))
    return out


def test_noalloc_equals_workspace_call_twice(qe, oracle):
    # first a 512 x 768 layer, then a smaller, ragged one: the second call
    # reuses the scratch the first one left behind
    for q, p, bits, sweeps, block in ((512, 768, 4, 4, 128), (77, 200, 3, 3, 64)):
        print(f"[noalloc] {q}x{p} bits={bits} sweeps={sweeps} block={block}", flush=True)
        W, S32, scale, zero = _layer(oracle, q, p, q + p, bits)
        ws_run, na_run = _both(qe, W, S32, scale, zero, bits, sweeps, block)
        for a, b in zip(ws_run[:4], na_run[:4]):
            assert np.array_equal(a, b)
        assert na_run[4] == 0
        # and both within the oracle's bar on the final objective
        ref = oracle.cd(W, S32.astype(np.float64), bits, scale, zero, sweeps)
        assert na_run[3][-1] == pytest.approx(ref.obj[-1], rel=1e-4)


def test_noalloc_status_reports_and_clears(qe, oracle):
    q, p = 16, 40
    W = synth.gaussian((q, p), seed=26)
    S = np.eye(p, dtype=np.float32)
    S[7, 7] = 0.0
    Wd, Sd = dev(W), dev(S)
    Wh = torch.empty_like(Wd)
    codes = torch.zeros((q, p), dtype=torch.uint8, device="cuda")
    R = torch.empty_like(Wd)
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    one = dev(np.ones(q, np.float32))
    zero = dev(np.zeros(q, np.float32))
    qe.cd_sweep_noalloc(Wd, Sd, 4, one, zero, Wh, codes, R, 1, status=status)
    torch.cuda.synchronize()
    assert int(host(status)[0]) == qe.QE_ERR_DIAG
    # the next call starts from a clear status word
    W2, S32, scale, zero2 = _layer(oracle, 64, 96, 5, 4)
    ws_run, na_run = _both(qe, W2, S32, scale, zero2, 4, 2, 0)
    assert na_run[4] == 0
    for a, b in zip(ws_run[:4], na_run[:4]):
        assert np.array_equal(a, b)


def test_noalloc_rejects_sizes_beyond_its_scratch(qe):
    """A layer whose scratch would exceed the fixed array is refused with
    QE_ERR_TOO_LARGE before anything is enqueued (outputs untouched)."""
    q, p = 40000, 4096
    assert qe.cd_workspace_size(q, p, 0) > qe.QE_NOALLOC_SCRATCH_BYTES
    W = torch.zeros((q, p), dtype=torch.float32, device="cuda")
    S = torch.eye(p, dtype=torch.float32, device="cuda")
    Wh = torch.full((q, p), 7.0, dtype=torch.float32, device="cuda")
    codes = torch.zeros((q, p), dtype=torch.uint8, device="cuda")
    sc = torch.ones(q, dtype=torch.float32, device="cuda")
    with pytest.raises(qe.QEError) as e:
        qe.cd_sweep_noalloc(W, S, 4, sc, torch.zeros_like(sc), Wh, codes, W, 1)
    assert e.value.code == qe.QE_ERR_TOO_LARGE
    torch.cuda.synchronize()
    assert bool(torch.all(Wh == 7.0))


def test_noalloc_call_replayed_from_a_graph(qe, oracle):
    q, p, bits, sweeps = 256, 384, 4, 3
    W = synth.gaussian((q, p), seed=41, std=0.02)
    X = synth.correlated_activations(p, 1024, 0.9, 41, out_channels=8, out_mult=20.0)
    S32 = oracle.damp(oracle.gram(X), 0.01).astype(np.float32)
    scale, zero = oracle.grid_minmax(W, bits)
    Wd, Sd, sc, ze = dev(W), dev(S32), dev(scale), dev(zero)

    def buffers():
        return (torch.empty_like(Wd), torch.zeros((q, p), dtype=torch.uint8, device="cuda"),
                torch.empty_like(Wd), torch.zeros(sweeps, dtype=torch.float64, device="cuda"),
                torch.full((1,), -1, dtype=torch.int32, device="cuda"))

    # eager call first (also where the scratch's address is looked up on this GPU)
    Wh, codes, R, obj, st = buffers()
    qe.cd_sweep_noalloc(Wd, Sd, bits, sc, ze, Wh, codes, R, sweeps, obj=obj, status=st)
    torch.cuda.synchronize()
    ref = [host(x) for x in (Wh, codes, R, obj, st)]
    assert ref[4][0] == 0

    # one call recorded (QE_INIT_FROM_W: every replay starts again from What = W)
    Wh2, codes2, R2, obj2, st2 = buffers()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        qe.cd_sweep_noalloc(Wd, Sd, bits, sc, ze, Wh2, codes2, R2, sweeps, obj=obj2, status=st2)
    torch.cuda.synchronize()
    for rep in range(3):
        # the program's own eager work between replays: overwrite every output
        Wh2.fill_(1.0)
        codes2.fill_(7)
        R2.fill_(-1.0)
        obj2.fill_(0.0)
        st2.fill_(-1)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = [host(x) for x in (Wh2, codes2, R2, obj2, st2)]
        for name, a, b in zip(("What", "codes", "R", "objective", "status"), ref, got):
            assert np.array_equal(a, b), f"replay {rep}: {name}"
