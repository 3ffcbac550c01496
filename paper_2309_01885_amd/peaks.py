"""Peak checks for the roofline denominators (libqe_peak.so, built beside
libqe.so from peak/peak.hip): matrix-core throughput of the bf16, fp16 and
fp32 MFMA instructions the products use, in register-only loops; the engine clock
under that load; and an HBM copy.  The vendor peaks stay the roofline
denominators; these say how much of them this chip sustains."""
import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libqe_peak.so")

BLOCKS = 512            # two 256-thread workgroups per CU on 256 CUs
COPY_SHAPES = ((1024, 0), (2048, 0), (4096, 1), (16384, 1))   # (workgroups, chunked)
_lib = None


def load():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built (run __graft_entry__.build())")
        lib = ctypes.CDLL(LIB_PATH)
        vp, i = ctypes.c_void_p, ctypes.c_int
        for f, args in (("qpk_mfma_bf16", [vp, i, i, vp]), ("qpk_mfma_f16", [vp, i, i, vp]),
                        ("qpk_mfma_f32", [vp, i, i, vp]),
                        ("qpk_clock", [vp, vp, i, i, vp]),
                        ("qpk_copy", [vp, vp, ctypes.c_size_t, i, i, vp])):
            getattr(lib, f).argtypes = args
            getattr(lib, f).restype = ctypes.c_int
        _lib = lib
    return _lib


def _timed(torch, launch, reps=3):
    """Best of `reps` launches (after one warm-up), seconds, on the current stream."""
    launch()
    best = None
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        launch()
        e1.record()
        e1.synchronize()
        t = e0.elapsed_time(e1) * 1e-3
        best = t if best is None else min(best, t)
    return best


def _ok(rc, name):
    if rc != 0:
        raise RuntimeError(f"{name} failed with status {rc}")


def measure(torch, bf16_iters=4000, f32_iters=2000, copy_bytes=1 << 30):
    lib = load()
    dev = torch.device("cuda", torch.cuda.current_device())
    st = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    out = torch.empty(BLOCKS * 256, dtype=torch.float32, device=dev)
    t_bf = _timed(torch, lambda: _ok(lib.qpk_mfma_bf16(out.data_ptr(), BLOCKS, bf16_iters, st),
                                     "qpk_mfma_bf16"))
    t_f16 = _timed(torch, lambda: _ok(lib.qpk_mfma_f16(out.data_ptr(), BLOCKS, bf16_iters, st),
                                      "qpk_mfma_f16"))
    t_f32 = _timed(torch, lambda: _ok(lib.qpk_mfma_f32(out.data_ptr(), BLOCKS, f32_iters, st),
                                      "qpk_mfma_f32"))
    waves_iters = BLOCKS * 4 * 16           # waves x MFMAs per iteration
    bf_tf = waves_iters * bf16_iters * 2 * 32 * 32 * 16 / t_bf / 1e12
    f16_tf = waves_iters * bf16_iters * 2 * 32 * 32 * 16 / t_f16 / 1e12
    f32_tf = waves_iters * f32_iters * 2 * 32 * 32 * 2 / t_f32 / 1e12
    clk = torch.zeros(BLOCKS * 4 * 2, dtype=torch.int64, device=dev)
    _ok(lib.qpk_clock(out.data_ptr(), clk.data_ptr(), BLOCKS, bf16_iters, st), "qpk_clock")
    c = clk.view(-1, 2).double().cpu()
    ghz = float((c[:, 0] / (c[:, 1] / 100e6)).median()) / 1e9
    n16 = copy_bytes // 16
    src = torch.ones(n16 * 4, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    t_cp = min(_timed(torch, lambda: _ok(lib.qpk_copy(src.data_ptr(), dst.data_ptr(), n16, b, ch,
                                                      st), "qpk_copy"))
               for b, ch in COPY_SHAPES)
    ok = bool(torch.equal(src, dst))
    del src, dst
    return {"mfma_bf16_tflops": bf_tf, "mfma_f16_tflops": f16_tf, "mfma_f32_tflops": f32_tf,
            "engine_clock_ghz_under_mfma": ghz, "copy_gbps": 2 * n16 * 16 / t_cp / 1e9,
            "copy_checked": ok,
            "method": (f"register-only v_mfma_f32_32x32x16_bf16 / _f16 / v_mfma_f32_32x32x2f32 loops, "
                       f"{BLOCKS} workgroups of 4 waves, 4 accumulators a wave; clock from "
                       f"s_memtime over s_memrealtime; copy of {copy_bytes >> 20} MiB, best of "
                       f"(workgroups, chunked) in {COPY_SHAPES}; best of 3")}
